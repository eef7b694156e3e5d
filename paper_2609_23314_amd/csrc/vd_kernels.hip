// HIP kernels of the ValueDiff eviction pass for gfx950 (MI355X).
//
// One workgroup of 1024 threads (16 wave64s) owns one unit (sequence, layer,
// KV head).  The pass is bound by HBM bandwidth: it streams the unit's value
// rows once, with 16-byte loads per lane and a row spread over LPR lanes
// (LPR = row bytes / 16; 16 lanes for a 128-channel bf16 row), reduces each
// row over its lanes with DPP, and keeps everything else (scores, selection,
// move lists, optionally the newly appended rows) in LDS.
//
//   mean    fp64 column sums of the rows not yet summed (all n, or only the
//           appended rows when the caller keeps a running sum), reduced in a
//           fixed order                                     (Sec. 3.2, Eq. vd)
//   score   fp32, one DPP row reduction per row (two for Dir)  (Sec. 3.2)
//   select  radix select of the N-th largest fp32 score on its order-
//           preserving uint32 key, ties to the lower slot; a single block
//           argmin when exactly one token goes (decode)  (Sec. 2.1, Eq. eviction)
//   gather  slot reuse: evicted slots below N, ascending, receive the kept
//           slots at or above N, ascending; only those rows move
//
// No MFMA: nothing here is a dense contraction.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "vd_launch.h"

namespace vd {
namespace {

constexpr int NT = kBlock;
constexpr int NW = kWaves;
constexpr int kUnroll = 8;  // 16-byte loads in flight per lane in the row streams

// ---------------------------------------------------------------- elements

template <int DT> struct Elem;
template <> struct Elem<0> {  // bfloat16: the upper half of a binary32
    static constexpr int BYTES = 2, EPL = 8;
    __device__ static __forceinline__ void unpack(const uint4 w, float *x) {
        x[0] = __uint_as_float(w.x << 16); x[1] = __uint_as_float(w.x & 0xFFFF0000u);
        x[2] = __uint_as_float(w.y << 16); x[3] = __uint_as_float(w.y & 0xFFFF0000u);
        x[4] = __uint_as_float(w.z << 16); x[5] = __uint_as_float(w.z & 0xFFFF0000u);
        x[6] = __uint_as_float(w.w << 16); x[7] = __uint_as_float(w.w & 0xFFFF0000u);
    }
};
template <> struct Elem<1> {  // fp32
    static constexpr int BYTES = 4, EPL = 4;
    __device__ static __forceinline__ void unpack(const uint4 w, float *x) {
        x[0] = __uint_as_float(w.x); x[1] = __uint_as_float(w.y);
        x[2] = __uint_as_float(w.z); x[3] = __uint_as_float(w.w);
    }
};

template <int DT, int D> struct Shape {
    static constexpr int EPL = Elem<DT>::EPL;
    static constexpr int ROWB = D * Elem<DT>::BYTES;  // bytes per row
    static constexpr int LPR = ROWB / 16;             // lanes per row
    static constexpr int RPW = 64 / LPR;              // rows per wave instruction
    static constexpr int GROUPS = NW * RPW;           // row groups per workgroup
    static_assert(LPR >= 1 && LPR <= 64 && 64 % LPR == 0, "unsupported row shape");
};

// ---------------------------------------------------------------- lane utils

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

template <int CTRL> __device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over the LPR lanes holding one row; every lane of the group receives the
// same bits (each step adds a pair of equal operands in swapped order).
template <int LPR> __device__ __forceinline__ float row_sum(float x) {
    if constexpr (LPR >= 2) x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
    if constexpr (LPR >= 4) x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
    if constexpr (LPR >= 8) x += dpp<0x141>(x);  // row_half_mirror
    if constexpr (LPR >= 16) x += dpp<0x140>(x); // row_mirror
    if constexpr (LPR >= 32) x += __shfl_xor(x, 16);
    if constexpr (LPR >= 64) x += __shfl_xor(x, 32);
    return x;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    for (int o = 32; o > 0; o >>= 1) x = min(x, (uint32_t)__shfl_xor((int)x, o));
    return x;
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    for (int o = 32; o > 0; o >>= 1) x = max(x, (uint32_t)__shfl_xor((int)x, o));
    return x;
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t y = __shfl_xor((unsigned long long)x, o);
        x = y < x ? y : x;
    }
    return x;
}

// Order-preserving map of an fp32 value onto uint32 (-0 taken as +0).
__device__ __forceinline__ uint32_t orderable(float f) {
    uint32_t b = __float_as_uint(f);
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive rank of `flag` among the block's threads in thread order, and the
// block-wide count.  Two barriers; `wsum` holds NW entries.
__device__ __forceinline__ uint32_t block_rank(bool flag, uint32_t *wsum, uint32_t &total) {
    const uint64_t m = __ballot(flag);
    const int lane = lane_id(), w = wave_id();
    const uint32_t in_wave = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[w] = __popcll(m);
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const uint32_t c = wsum[i];
        before += (i < w) ? c : 0u;
        tot += c;
    }
    __syncthreads();
    total = tot;
    return before + in_wave;
}

// ---------------------------------------------------------------- row streams

// Streams `count` rows: element e (0 <= e < count) is row row_of(e), fetched
// 16 bytes per lane by fetch(row, chunk); body(e, valid, data) runs on every
// lane (lanes past the end see zeros and valid == false), so DPP reductions
// inside body always see full row groups.  kUnroll loads are issued before the
// first use.
template <int DT, int D, typename RowOf, typename Fetch, typename Body>
__device__ __forceinline__ void for_rows(int count, RowOf row_of, Fetch fetch, Body body) {
    using S = Shape<DT, D>;
    const int lane = lane_id(), w = wave_id();
    const int q = lane / S::LPR, cl = lane % S::LPR;
    constexpr int STEP = S::GROUPS * kUnroll;
    for (int e0 = 0; e0 < count; e0 += STEP) {
        uint4 buf[kUnroll];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int e = e0 + (k * NW + w) * S::RPW + q;
            buf[k] = e < count ? fetch(row_of(e), cl) : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int e = e0 + (k * NW + w) * S::RPW + q;
            body(e, e < count, buf[k]);
        }
    }
}

// Column sums of per-lane fp64 partials (each lane holds EPL columns of its
// chunk) into out[0..D) in LDS; fixed reduction order.  `red` holds NW*D doubles.
template <int DT, int D>
__device__ __forceinline__ void block_col_sums(double *acc, double *red, double *out) {
    using S = Shape<DT, D>;
#pragma unroll
    for (int o = S::LPR; o < 64; o <<= 1)
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) acc[i] += __shfl_xor(acc[i], o);
    const int lane = lane_id(), w = wave_id();
    if (lane < S::LPR)
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) red[w * D + lane * S::EPL + i] = acc[i];
    __syncthreads();
    for (int t = threadIdx.x; t < D; t += NT) {
        double s = 0.0;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) s += red[ww * D + t];
        out[t] = s;
    }
    __syncthreads();
}

// ---------------------------------------------------------------- selection

struct Threshold {
    uint32_t key;      // key of the N-th largest score
    int need;          // how many keys equal to `key` are kept (the lowest slots)
    int count_eq;      // how many keys equal `key`
};

// Radix select of the N-th largest of keys[0..n) (1 <= N < n), MSB first,
// 8-bit digits starting at the highest bit in which the keys differ.
__device__ Threshold radix_select(const uint32_t *keys, int n, int N, LdsHead &H) {
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    for (int j = threadIdx.x; j < n; j += NT) {
        const uint32_t k = keys[j];
        kmin = min(kmin, k);
        kmax = max(kmax, k);
    }
    kmin = wave_min_u32(kmin);
    kmax = wave_max_u32(kmax);
    if (lane_id() == 0) {
        H.bc[wave_id()] = kmin;
        H.bc[32 + wave_id()] = kmax;
    }
    __syncthreads();
    kmin = H.bc[0];
    kmax = H.bc[32];
#pragma unroll
    for (int i = 1; i < NW; ++i) {
        kmin = min(kmin, H.bc[i]);
        kmax = max(kmax, H.bc[32 + i]);
    }
    __syncthreads();
    if (kmin == kmax) return Threshold{kmin, N, n};

    const int hb = 31 - __clz(kmin ^ kmax);
    uint32_t prefix = hb == 31 ? 0u : (kmin & ~((2u << hb) - 1u));
    int need = N;
    int top = hb;
    int count_in_bin = 0;
    for (;;) {
        const int width = top + 1 < 8 ? top + 1 : 8;
        const int shift = top + 1 - width;
        const uint32_t hi_mask = top == 31 ? 0u : ~((2u << top) - 1u);
        const uint32_t dmask = (1u << width) - 1u;
        for (int i = threadIdx.x; i < 256; i += NT) H.hist[i] = 0u;
        __syncthreads();
        for (int j = threadIdx.x; j < n; j += NT) {
            const uint32_t k = keys[j];
            if ((k & hi_mask) == prefix) atomicAdd(&H.hist[(k >> shift) & dmask], 1u);
        }
        __syncthreads();
        if (wave_id() == 0) {
            // lane l owns bins 4l..4l+3; find bin b with above(b) < need <= above(b) + hist[b]
            const int l = lane_id();
            const uint32_t h0 = H.hist[4 * l], h1 = H.hist[4 * l + 1];
            const uint32_t h2 = H.hist[4 * l + 2], h3 = H.hist[4 * l + 3];
            const uint32_t local = h0 + h1 + h2 + h3;
            uint32_t suf = local;  // inclusive suffix sum over lanes
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t t = __shfl_down(suf, o);
                if (l + o < 64) suf += t;
            }
            uint32_t above = suf - local;
            const uint32_t hh[4] = {h0, h1, h2, h3};
            const uint32_t un = (uint32_t)need;
#pragma unroll
            for (int t = 3; t >= 0; --t) {
                if (above < un && un <= above + hh[t]) {
                    H.bc[64] = 4u * l + t;
                    H.bc[65] = above;
                    H.bc[66] = hh[t];
                }
                above += hh[t];
            }
        }
        __syncthreads();
        const uint32_t b = H.bc[64];
        need -= (int)H.bc[65];
        count_in_bin = (int)H.bc[66];
        __syncthreads();
        prefix |= b << shift;
        if (shift == 0) break;
        top = shift - 1;
    }
    return Threshold{prefix, need, count_in_bin};
}

// Walks slots [0, n) in block-sized chunks and decides keep(j) from the
// threshold; appends evicted slots (ascending) to evl and kept slots >= N
// (ascending) to mvl; writes keep_out if given.  Returns the mover count.
__device__ int build_lists(const uint32_t *keys, int n, int N, const Threshold &th,
                           uint32_t *evl, int evict_cap, uint32_t *mvl, int move_cap,
                           uint8_t *keep_out, LdsHead &H) {
    uint32_t eq_off = 0, ev_off = 0, mv_off = 0;
    const bool rank_eq = th.count_eq != th.need;
    for (int base = 0; base < n; base += NT) {
        const int j = base + threadIdx.x;
        const bool valid = j < n;
        const uint32_t k = valid ? keys[j] : 0u;
        const bool gt = valid && k > th.key;
        const bool eq = valid && k == th.key;
        bool keep = gt || eq;
        if (rank_eq) {
            uint32_t tot;
            const uint32_t r = block_rank(eq, H.bc, tot) + eq_off;
            eq_off += tot;
            keep = gt || (eq && r < (uint32_t)th.need);
        }
        uint32_t tot_ev, tot_mv;
        const uint32_t rev = block_rank(valid && !keep, H.bc, tot_ev) + ev_off;
        const uint32_t rmv = block_rank(valid && keep && j >= N, H.bc, tot_mv) + mv_off;
        if (valid && !keep && rev < (uint32_t)evict_cap) evl[rev] = (uint32_t)j;
        if (valid && keep && j >= N && rmv < (uint32_t)move_cap) mvl[rmv] = (uint32_t)j;
        if (keep_out && valid) keep_out[j] = keep ? 1 : 0;
        ev_off += tot_ev;
        mv_off += tot_mv;
    }
    __syncthreads();
    return (int)mv_off;
}

// ---------------------------------------------------------------- the pass

template <int DT, int D, int VAR>
__global__ void __launch_bounds__(NT) step_kernel(const UnitParams p) {
    using S = Shape<DT, D>;
    using E = Elem<DT>;
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    uint32_t *keys = reinterpret_cast<uint32_t *>(lds + p.off_keys);
    double *red = reinterpret_cast<double *>(lds + p.off_keys);  // aliases keys
    uint32_t *evl = reinterpret_cast<uint32_t *>(lds + p.off_lists);
    uint32_t *mvl = evl + p.evict_cap;
    unsigned char *stash = lds + p.off_stash;

    const int ul = blockIdx.x;
    const int sl = ul / (p.num_layers * p.num_kv_heads);
    const int layer = (ul / p.num_kv_heads) % p.num_layers;
    const int head = ul % p.num_kv_heads;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.n[sl], N = p.N[sl];
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    const char *vb = p.v + off;
    const int64_t ss = p.s_slot;
    const int64_t cap = p.capacity;
    const int lane = lane_id();
    const int cl = lane % S::LPR;

    const bool score_mode = p.mode == kModeScore;
    double *st = score_mode ? nullptr : (p.running_sum ? p.running_sum + u * (D + 1) : nullptr);
    const bool evict = !score_mode && n > N;
    float *scores_out = p.scores ? p.scores + u * cap : nullptr;
    uint8_t *keep_out = p.keep ? p.keep + u * cap : nullptr;

    if (n <= 0) {
        if (st) {
            for (int t = threadIdx.x; t <= D; t += NT) st[t] = 0.0;
        }
        return;
    }
    const bool need_scores = score_mode || evict || scores_out;
    if (!need_scores && !st) {
        for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = 1;
        return;
    }

    // ---- mean: sum the rows not yet summed (Sec. 3.2, Eq. vd) ----
    int count = 0;
    if (st) {
        const double c = st[D];
        count = (c >= 0.0 && c <= (double)n && c == (double)(int)c) ? (int)c : 0;
    }
    const int fresh = n - count;
    const bool stashed = fresh <= p.stash_rows;
    auto gfetch = [&](int r, int c) -> uint4 {
        return *reinterpret_cast<const uint4 *>(vb + (int64_t)r * ss + c * 16);
    };
    auto sfetch = [&](int r, int c) -> uint4 {
        return *reinterpret_cast<const uint4 *>(stash + (int64_t)(r - count) * S::ROWB + c * 16);
    };
    {
        double acc[S::EPL];
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) acc[i] = 0.0;
        for_rows<DT, D>(fresh, [&](int e) { return count + e; }, gfetch,
                        [&](int e, bool valid, uint4 w) {
                            float x[S::EPL];
                            E::unpack(w, x);
#pragma unroll
                            for (int i = 0; i < S::EPL; ++i) acc[i] += (double)x[i];
                            if (stashed && valid)
                                *reinterpret_cast<uint4 *>(stash + (int64_t)e * S::ROWB + cl * 16) = w;
                        });
        block_col_sums<DT, D>(acc, red, H.sum);
    }
    for (int t = threadIdx.x; t < D; t += NT) {
        const double s = (count > 0 ? st[t] : 0.0) + H.sum[t];
        H.sum[t] = s;
        H.mean[t] = (float)(s / (double)n);
    }
    __syncthreads();
    bool mean_zero = false;
    if constexpr (VAR == 1) {
        if (wave_id() == 0) {
            float a = 0.f;
            for (int t = lane; t < D; t += 64) a += H.mean[t] * H.mean[t];
            for (int o = 32; o > 0; o >>= 1) a += __shfl_xor(a, o);
            if (lane == 0) H.bc[0] = __float_as_uint(a);
        }
        __syncthreads();
        const float mn2 = __uint_as_float(H.bc[0]);
        const float mn = sqrtf(mn2);
        mean_zero = !(mn2 > 0.f);
        for (int t = threadIdx.x; t < D; t += NT) H.udir[t] = mean_zero ? 0.f : H.mean[t] / mn;
        __syncthreads();
    }
    if (score_mode && p.mean_out)
        for (int t = threadIdx.x; t < D; t += NT) p.mean_out[u * D + t] = H.mean[t];

    // ---- scores (Sec. 3.2) ----
    const bool amode = evict && n == N + 1;  // decode: exactly one token goes
    uint64_t best = ~0ull;                    // (key << 32) | ~slot: min = lowest score, highest slot
    if (need_scores) {
        float m[S::EPL];
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) m[i] = (VAR == 1 ? H.udir : H.mean)[cl * S::EPL + i];
        const bool to_lds = evict && !amode;
        auto on_row = [&](int r, bool valid, uint4 w) {
            float x[S::EPL];
            E::unpack(w, x);
            float s;
            if constexpr (VAR == 0) {  // L2: ||v - v_bar||
                float a = 0.f;
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) {
                    const float t = x[i] - m[i];
                    a = fmaf(t, t, a);
                }
                s = sqrtf(row_sum<S::LPR>(a));
            } else if constexpr (VAR == 2) {  // Norm: ||v||
                float a = 0.f;
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) a = fmaf(x[i], x[i], a);
                s = sqrtf(row_sum<S::LPR>(a));
            } else {  // Dir: 1 - cos = ||v/|v| - v_bar/|v_bar| ||^2 / 2
                float a = 0.f;
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) a = fmaf(x[i], x[i], a);
                const float nv2 = row_sum<S::LPR>(a);
                const bool ok = nv2 > 0.f && !mean_zero;
                const float inv = ok ? 1.0f / sqrtf(nv2) : 0.f;
                float b = 0.f;
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) {
                    const float t = fmaf(x[i], inv, -m[i]);
                    b = fmaf(t, t, b);
                }
                const float half = 0.5f * row_sum<S::LPR>(b);
                s = ok ? half : 1.0f;
            }
            if (cl == 0 && valid) {
                const uint32_t key = orderable(s);
                if (to_lds) keys[r] = key;
                if (amode) {
                    const uint64_t c = ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)r);
                    best = c < best ? c : best;
                }
                if (scores_out) scores_out[r] = s;
            }
        };
        for_rows<DT, D>(count, [](int e) { return e; }, gfetch,
                        [&](int e, bool valid, uint4 w) { on_row(e, valid, w); });
        if (stashed)
            for_rows<DT, D>(fresh, [&](int e) { return count + e; }, sfetch,
                            [&](int e, bool valid, uint4 w) { on_row(count + e, valid, w); });
        else
            for_rows<DT, D>(fresh, [&](int e) { return count + e; }, gfetch,
                            [&](int e, bool valid, uint4 w) { on_row(count + e, valid, w); });
    }
    __syncthreads();
    if (score_mode) return;

    // ---- select (Sec. 2.1, Eq. eviction) ----
    int n_moves = 0;
    if (evict) {
        if (amode) {
            best = wave_min_u64(best);
            if (lane == 0) {
                H.bc[2 * wave_id()] = (uint32_t)(best >> 32);
                H.bc[2 * wave_id() + 1] = (uint32_t)best;
            }
            __syncthreads();
            uint64_t b = ~0ull;
#pragma unroll
            for (int i = 0; i < NW; ++i) {
                const uint64_t c = ((uint64_t)H.bc[2 * i] << 32) | H.bc[2 * i + 1];
                b = c < b ? c : b;
            }
            const int victim = (int)(0xFFFFFFFFu - (uint32_t)b);
            __syncthreads();
            if (threadIdx.x == 0) {
                evl[0] = (uint32_t)victim;
                mvl[0] = (uint32_t)N;  // slot N = n - 1 is kept unless it is the victim
            }
            n_moves = victim < N ? 1 : 0;
            for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = j == victim ? 0 : 1;
            __syncthreads();
        } else {
            const Threshold th = radix_select(keys, n, N, H);
            n_moves = build_lists(keys, n, N, th, evl, p.evict_cap, mvl, p.move_cap, keep_out, H);
        }
    } else {
        for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = 1;
    }

    // ---- running sum: remove the evicted rows ----
    if (st) {
        if (evict) {
            double acc[S::EPL];
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) acc[i] = 0.0;
            auto body = [&](int, bool, uint4 w) {
                float x[S::EPL];
                E::unpack(w, x);
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) acc[i] += (double)x[i];
            };
            auto fetch = [&](int r, int c) -> uint4 {
                return (stashed && r >= count) ? sfetch(r, c) : gfetch(r, c);
            };
            for_rows<DT, D>(n - N, [&](int e) { return (int)evl[e]; }, fetch, body);
            // red aliases keys, which the lists no longer need
            block_col_sums<DT, D>(acc, red, H.sum_ev);
            for (int t = threadIdx.x; t < D; t += NT) st[t] = H.sum[t] - H.sum_ev[t];
            if (threadIdx.x == 0) st[D] = (double)N;
        } else {
            for (int t = threadIdx.x; t < D; t += NT) st[t] = H.sum[t];
            if (threadIdx.x == 0) st[D] = (double)n;
        }
        __syncthreads();
    }

    // ---- gather with slot reuse ----
    if (n_moves > 0) {
        char *kb = p.k ? p.k + off : nullptr;
        char *vw = p.v + off;
        int32_t *pos = p.pos ? p.pos + u * cap : nullptr;
        const int lane_q = lane / S::LPR;
        const int g = wave_id() * S::RPW + lane_q;  // row group of this lane
        for (int e = g; e < n_moves; e += S::GROUPS) {
            const int dst = (int)evl[e];
            const int src = (int)mvl[e];
            if (kb) {
                const uint4 kv = *reinterpret_cast<const uint4 *>(kb + (int64_t)src * ss + cl * 16);
                *reinterpret_cast<uint4 *>(kb + (int64_t)dst * ss + cl * 16) = kv;
            }
            const uint4 vv = (stashed && src >= count) ? sfetch(src, cl) : gfetch(src, cl);
            *reinterpret_cast<uint4 *>(vw + (int64_t)dst * ss + cl * 16) = vv;
            if (pos && cl == 0) pos[dst] = pos[src];
        }
    }
}

// Standalone selection: scores (global) -> keep mask.
__global__ void __launch_bounds__(NT) select_kernel(const UnitParams p) {
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    uint32_t *keys = reinterpret_cast<uint32_t *>(lds + p.off_keys);
    const int ul = blockIdx.x;
    const int sl = ul / (p.num_layers * p.num_kv_heads);
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.n[sl], N = p.N[sl];
    const int64_t cap = p.capacity;
    const float *sc = p.scores_in + u * cap;
    uint8_t *keep = p.keep + u * cap;
    if (n <= N) {
        for (int j = threadIdx.x; j < n; j += NT) keep[j] = 1;
        return;
    }
    for (int j = threadIdx.x; j < n; j += NT) keys[j] = orderable(sc[j]);
    __syncthreads();
    const Threshold th = radix_select(keys, n, N, H);
    const bool rank_eq = th.count_eq != th.need;
    uint32_t eq_off = 0;
    for (int base = 0; base < n; base += NT) {
        const int j = base + threadIdx.x;
        const bool valid = j < n;
        const uint32_t k = valid ? keys[j] : 0u;
        const bool gt = valid && k > th.key;
        const bool eq = valid && k == th.key;
        bool kp = gt || eq;
        if (rank_eq) {
            uint32_t tot;
            const uint32_t r = block_rank(eq, H.bc, tot) + eq_off;
            eq_off += tot;
            kp = gt || (eq && r < (uint32_t)th.need);
        }
        if (valid) keep[j] = kp ? 1 : 0;
    }
}

// Standalone gather from a keep mask.
template <int DT, int D>
__global__ void __launch_bounds__(NT) compact_kernel(const UnitParams p) {
    using S = Shape<DT, D>;
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    uint32_t *holes = reinterpret_cast<uint32_t *>(lds + p.off_lists);
    uint32_t *movers = holes + p.evict_cap;
    const int ul = blockIdx.x;
    const int sl = ul / (p.num_layers * p.num_kv_heads);
    const int layer = (ul / p.num_kv_heads) % p.num_layers;
    const int head = ul % p.num_kv_heads;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.n[sl], N = p.N[sl];
    if (n <= N) return;
    const int64_t cap = p.capacity;
    const uint8_t *keep = p.keep_in + u * cap;
    uint32_t h_off = 0, m_off = 0;
    for (int base = 0; base < n; base += NT) {
        const int j = base + threadIdx.x;
        const bool valid = j < n;
        const bool kp = valid && keep[j] != 0;
        uint32_t th, tm;
        const uint32_t rh = block_rank(valid && j < N && !kp, H.bc, th) + h_off;
        const uint32_t rm = block_rank(kp && j >= N, H.bc, tm) + m_off;
        if (valid && j < N && !kp && rh < (uint32_t)p.evict_cap) holes[rh] = (uint32_t)j;
        if (kp && j >= N && rm < (uint32_t)p.move_cap) movers[rm] = (uint32_t)j;
        h_off += th;
        m_off += tm;
    }
    __syncthreads();
    int moves = (int)min(h_off, m_off);
    moves = min(moves, min(p.evict_cap, p.move_cap));
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    char *kb = p.k ? p.k + off : nullptr;
    char *vb = p.v + off;
    int32_t *pos = p.pos ? p.pos + u * cap : nullptr;
    const int64_t ss = p.s_slot;
    const int lane = lane_id();
    const int cl = lane % S::LPR;
    const int g = wave_id() * S::RPW + lane / S::LPR;
    for (int e = g; e < moves; e += S::GROUPS) {
        const int dst = (int)holes[e];
        const int src = (int)movers[e];
        if (kb) {
            const uint4 kv = *reinterpret_cast<const uint4 *>(kb + (int64_t)src * ss + cl * 16);
            *reinterpret_cast<uint4 *>(kb + (int64_t)dst * ss + cl * 16) = kv;
        }
        const uint4 vv = *reinterpret_cast<const uint4 *>(vb + (int64_t)src * ss + cl * 16);
        *reinterpret_cast<uint4 *>(vb + (int64_t)dst * ss + cl * 16) = vv;
        if (pos && cl == 0) pos[dst] = pos[src];
    }
}

template <int DT, int D> void *step_kernel_for(int variant) {
    switch (variant) {
        case 0: return reinterpret_cast<void *>(&step_kernel<DT, D, 0>);
        case 1: return reinterpret_cast<void *>(&step_kernel<DT, D, 1>);
        case 2: return reinterpret_cast<void *>(&step_kernel<DT, D, 2>);
    }
    return nullptr;
}

template <int DT> void *step_kernel_for(int head_dim, int variant) {
    switch (head_dim) {
        case 64: return step_kernel_for<DT, 64>(variant);
        case 128: return step_kernel_for<DT, 128>(variant);
        case 256: return step_kernel_for<DT, 256>(variant);
    }
    return nullptr;
}

template <int DT> void *compact_kernel_for(int head_dim) {
    switch (head_dim) {
        case 64: return reinterpret_cast<void *>(&compact_kernel<DT, 64>);
        case 128: return reinterpret_cast<void *>(&compact_kernel<DT, 128>);
        case 256: return reinterpret_cast<void *>(&compact_kernel<DT, 256>);
    }
    return nullptr;
}

hipError_t launch(void *fn, int num_units, size_t lds_bytes, hipStream_t stream,
                  const UnitParams &p) {
    if (!fn) return hipErrorInvalidDeviceFunction;
    void *args[] = {const_cast<UnitParams *>(&p)};
    return hipLaunchKernel(fn, dim3(num_units), dim3(NT), args, lds_bytes, stream);
}

}  // namespace

hipError_t launch_step(const UnitParams &p, int num_units, int dtype, int head_dim,
                       int variant, size_t lds_bytes, hipStream_t stream) {
    void *fn = dtype == 0 ? step_kernel_for<0>(head_dim, variant)
                          : step_kernel_for<1>(head_dim, variant);
    return launch(fn, num_units, lds_bytes, stream, p);
}

hipError_t launch_select(const UnitParams &p, int num_units, size_t lds_bytes,
                         hipStream_t stream) {
    return launch(reinterpret_cast<void *>(&select_kernel), num_units, lds_bytes, stream, p);
}

hipError_t launch_compact(const UnitParams &p, int num_units, int dtype, int head_dim,
                          size_t lds_bytes, hipStream_t stream) {
    void *fn = dtype == 0 ? compact_kernel_for<0>(head_dim) : compact_kernel_for<1>(head_dim);
    return launch(fn, num_units, lds_bytes, stream, p);
}

}  // namespace vd
