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
//           fixed order; the first scoring tile is already in flight
//                                                        (Sec. 3.2, Eq. vd)
//   score   fp32, one DPP row reduction per row (two for Dir)  (Sec. 3.2)
//   select  the N-th largest fp32 score on its order-preserving uint32 key:
//           a histogram over the key range narrows it to one bin, whose few
//           keys one wave ranks exactly; ties go to the lower slot; a single
//           block argmin when exactly one token goes (decode)
//                                                 (Sec. 2.1, Eq. eviction)
//   gather  slot reuse: evicted slots below N, ascending, receive the kept
//           slots at or above N, ascending; only those rows move; the same
//           loop reads the evicted rows for the running-sum update
//
// A separate kernel, outside the pass, gives the key and value geometry of
// each unit (spread of the distances to the centroid, Sec. 3.1; bos-cosim,
// Sec. 4).
//
// The row stream is software-pipelined: chunk k of tile t+1 is requested as
// soon as chunk k of tile t is used, and every lane loads unconditionally
// (rows past the end are clamped to the last row and ignored).  The pass
// has no dense contraction and no MFMA; the fused decode attention's
// weighted sum of value rows for four query heads per KV head runs on the
// matrix cores (fp32 4 x 4 x 1 blocks), everything else on the vector ALUs.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "vd_launch.h"

// Device memory of the allocation-free fused decode step: its split partials
// live here instead of in a workspace of the caller's.  Every GPU the library
// runs on holds its own copy until the process ends, and every call on that
// GPU uses it (calls that overlap on one GPU race).  Host code never passes
// this name to a kernel: it takes the address hipGetSymbolAddress gives for
// the current device (vd::scratch_memory below).
static __device__ __align__(256) unsigned char scratch[vd::kScratchBytes];

#ifndef VD_DEBUG
#define VD_DEBUG 0
#endif
#if VD_DEBUG
// Debug builds: every index into a dynamically planned LDS region (keys and
// the second histogram, move lists, staged rows, fp64 reduction scratch, the
// FastCAOTE row buffer) is checked against the extent the host planned for it;
// a violation sets the site's bit here and the access is clamped to index 0.
// The host reads and clears the word (vd_debug_take_error_word).
__device__ unsigned int vd_debug_error_word;
#endif

namespace vd {
namespace {

// Sites of the LDS index checks (bit numbers of the debug error word).
enum : int { kSiteKeys = 0, kSiteHist = 1, kSiteEvl = 2, kSiteMvl = 3, kSiteStash = 4, kSiteRed = 5,
             kSiteRows = 6, kSiteLists = 7 };

// Index i into an LDS region of cap elements (plain i in release builds).
template <int SITE> __device__ __forceinline__ int lds_ix(int i, int cap) {
#if VD_DEBUG
    if ((unsigned)i >= (unsigned)cap) {
        atomicOr(&vd_debug_error_word, 1u << SITE);
        return 0;
    }
#else
    (void)cap;
#endif
    return i;
}

template <int V> struct IntC { static constexpr int value = V; };
template <bool V> struct BoolC { static constexpr bool value = V; };

constexpr int NT = kBlock;
constexpr int NW = kWaves;
constexpr int kUnroll = 4;  // 16-byte rows per lane in a staged-row tile and a gather batch
constexpr int kChunks = 2 * kUnroll;  // the pass kernel's row stream: one tile of 8 in flight
static_assert(NT == kBins, "the selection gives every thread one histogram bin");

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
    static constexpr int STEP = GROUPS * kUnroll;     // rows per tile
    static_assert(LPR >= 8 && LPR <= 64 && 64 % LPR == 0, "unsupported row shape");
};

// ---------------------------------------------------------------- lane utils

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }
__device__ __forceinline__ uint64_t lanes_below() { return (1ull << lane_id()) - 1ull; }

template <int CTRL> __device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
// Lane L of each 16-lane row to every lane of that row (row_newbcast).
template <int L> __device__ __forceinline__ float row_bcast(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x150 + L, 0xF, 0xF, false));
}
template <int L> __device__ __forceinline__ long row_bcast(long x) {
    return __builtin_amdgcn_update_dpp(0L, x, 0x150 + L, 0xF, 0xF, false);
}
// f(IntC<0>{}), ..., f(IntC<N-1>{})
template <int N, int I = 0, typename F> __device__ __forceinline__ void static_for(F &&f) {
    if constexpr (I < N) {
        f(IntC<I>{});
        static_for<N, I + 1>(f);
    }
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

// Sums of four rows at once: a[q] is this lane's partial sum of row q (chunk
// q of a tile), and each row spans the LPR lanes of one row group.  Two
// exchanges inside each quad leave every lane with a pair sum of one row,
// which is then summed over the lanes holding the same row; afterwards lane c
// of the group holds the full sum of row quad_row(c).  Five adds for four
// rows, against four per row one at a time.
__device__ __forceinline__ int quad_row(int c) { return ((c & 1) << 1) | ((c >> 1) & 1); }
template <int LPR> __device__ __forceinline__ float row_sums4(const float (&a)[4], int c) {
    const bool b0 = c & 1, b1 = (c >> 1) & 1;
    // lanes with bit 0 clear keep rows 0 and 1, the others rows 2 and 3
    const float k0 = b0 ? a[2] : a[0], k1 = b0 ? a[3] : a[1];
    const float g0 = b0 ? a[0] : a[2], g1 = b0 ? a[1] : a[3];
    const float p0 = k0 + dpp<0xB1>(g0);  // quad_perm [1,0,3,2]: lane ^ 1
    const float p1 = k1 + dpp<0xB1>(g1);
    // lanes with bit 1 clear keep the first of the two, the others the second
    float x = (b1 ? p1 : p0) + dpp<0x4E>(b1 ? p0 : p1);  // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (LPR == 8) x += __shfl_xor(x, 4);
    if constexpr (LPR >= 16) {
        x += dpp<0x124>(x);  // row_ror:4
        x += dpp<0x128>(x);  // row_ror:8
    }
    if constexpr (LPR >= 32) x += __shfl_xor(x, 16);
    if constexpr (LPR >= 64) x += __shfl_xor(x, 32);
    return x;
}

template <int CTRL, int ROW_MASK = 0xF>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROW_MASK, 0xF, false);
}
__device__ __forceinline__ uint32_t lane_u32(uint32_t x, int lane) {
    return (uint32_t)__builtin_amdgcn_readlane((int)x, lane);
}

// Wave-wide minimum / maximum: DPP inside each 16-lane row, then the four
// row results by readlane.  Every lane of the wave takes part.
template <int CTRL> __device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
    return ((uint64_t)dpp_u32<CTRL>((uint32_t)(x >> 32)) << 32) | dpp_u32<CTRL>((uint32_t)x);
}
__device__ __forceinline__ uint64_t lane_u64(uint64_t x, int lane) {
    return ((uint64_t)lane_u32((uint32_t)(x >> 32), lane) << 32) | lane_u32((uint32_t)x, lane);
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
    uint64_t y = dpp_u64<0xB1>(x);   // quad_perm [1,0,3,2]
    x = y < x ? y : x;
    y = dpp_u64<0x4E>(x);            // quad_perm [2,3,0,1]
    x = y < x ? y : x;
    y = dpp_u64<0x141>(x);           // row_half_mirror
    x = y < x ? y : x;
    y = dpp_u64<0x140>(x);           // row_mirror
    x = y < x ? y : x;
    const uint64_t a = lane_u64(x, 0), b = lane_u64(x, 16), c = lane_u64(x, 32), d = lane_u64(x, 48);
    const uint64_t ab = b < a ? b : a, cd = d < c ? d : c;
    return cd < ab ? cd : ab;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    x = min(x, dpp_u32<0xB1>(x));
    x = min(x, dpp_u32<0x4E>(x));
    x = min(x, dpp_u32<0x141>(x));
    x = min(x, dpp_u32<0x140>(x));
    return min(min(lane_u32(x, 0), lane_u32(x, 16)), min(lane_u32(x, 32), lane_u32(x, 48)));
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = max(x, dpp_u32<0xB1>(x));
    x = max(x, dpp_u32<0x4E>(x));
    x = max(x, dpp_u32<0x141>(x));
    x = max(x, dpp_u32<0x140>(x));
    return max(max(lane_u32(x, 0), lane_u32(x, 16)), max(lane_u32(x, 32), lane_u32(x, 48)));
}

// Inclusive prefix sum over the wave's lanes: shifts of 1, 2, 4, 8 inside
// each row (row_shr, zero fill), then rows 1 and 3 add lane 15 of the row
// before (row_bcast:15) and rows 2 and 3 add lane 31 (row_bcast:31).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
    x += dpp_u32<0x111>(x);
    x += dpp_u32<0x112>(x);
    x += dpp_u32<0x114>(x);
    x += dpp_u32<0x118>(x);
    x += dpp_u32<0x142, 0xA>(x);
    x += dpp_u32<0x143, 0xC>(x);
    return x;
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Row addresses are a workgroup-uniform base plus a 32-bit byte offset (the
// host checks that a unit's slab spans less than 4 GiB), so every access is a
// scalar-base load or store with one offset register per lane.
__device__ __forceinline__ uint32_t row_off(int r, uint32_t ss, int chunk) {
    return (uint32_t)r * ss + (uint32_t)chunk * 16u;
}

// Zero, produced by an empty asm that takes x: code using it cannot be
// scheduled before x is computed.
__device__ __forceinline__ uint32_t zero_after(float x) {
    uint32_t z = 0u;
    asm("" : "+v"(z) : "v"(x));
    return z;
}
template <int N> __device__ __forceinline__ uint32_t zero_after(const double (&x)[N]) {
    uint32_t z = 0u;
#pragma unroll
    for (int i = 0; i < N; ++i) asm("" : "+v"(z) : "v"(x[i]));
    return z;
}

// 16-byte load that bypasses cache retention: the value rows stream through once.
__device__ __forceinline__ uint4 load_stream(const char *base, uint32_t off) {
    const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(base + off));
    return make_uint4(t.x, t.y, t.z, t.w);
}

// 16-byte store that is not kept in the cache: moved rows are not read again here.
__device__ __forceinline__ void store_stream(char *base, uint32_t off, uint4 v) {
    u32x4 t;
    t.x = v.x; t.y = v.y; t.z = v.z; t.w = v.w;
    __builtin_nontemporal_store(t, reinterpret_cast<u32x4 *>(base + off));
}

// Square root and reciprocal square root of the scores: the hardware
// instructions (within one unit in the last place) without the exact-rounding
// fix-up sequence.  Subnormal inputs are scaled by 2^64 first, since the
// hardware units do not take them.  Every score of the library goes through
// these two, so the standalone and the fused paths agree bit for bit.
__device__ __forceinline__ float score_sqrt(float x) {
    const bool tiny = x < 1.17549435e-38f;  // below the smallest normal
    const float r = __builtin_amdgcn_sqrtf(tiny ? x * 18446744073709551616.0f : x);
    return tiny ? r * 2.3283064365386963e-10f : r;  // 2^-32
}
__device__ __forceinline__ float score_rsqrt(float x) {
    const bool tiny = x < 1.17549435e-38f;
    const float r = __builtin_amdgcn_rsqf(tiny ? x * 18446744073709551616.0f : x);
    return tiny ? r * 4294967296.0f : r;  // 2^32
}

// Order-preserving key of a score: scores are never negative (sums of squares
// and their roots, or half a squared distance), and for non-negative floats
// (+0 and -0 alike) setting the sign bit preserves the order.
__device__ __forceinline__ uint32_t score_key(float s) { return __float_as_uint(s) | 0x80000000u; }

// Score forms of the pass kernel: the scored rows are the value rows, or the
// key rows for a key-side score (the host hands the kernel K in V's place).
// kKeepSmallest is the norm with the order reversed (KeyNorm keeps the
// smallest norms): its key is the complement of the norm's, so that "keep the
// largest keys" and every tie rule stay as they are.
enum : int { kL2 = 0, kDir = 1, kNorm = 2, kKeepSmallest = 3 };
template <int VAR> __device__ __forceinline__ uint32_t key_of(float s) {
    return VAR == kKeepSmallest ? ~score_key(s) : score_key(s);
}
template <int VAR> __device__ __forceinline__ float score_of(uint32_t key) {
    return __uint_as_float((VAR == kKeepSmallest ? ~key : key) & 0x7FFFFFFFu);
}

// Order-preserving map of an fp32 value onto uint32 (-0 taken as +0).
__device__ __forceinline__ uint32_t orderable(float f) {
    uint32_t b = __float_as_uint(f);
    if (b == 0x80000000u) b = 0u;
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// x + (x of lane ^ 8, 16 or 32): each lane pair ends with the same bits.
template <int O> __device__ __forceinline__ double xor_sum(double x) {
    const unsigned long long b = __double_as_longlong(x);
    const unsigned lo = (unsigned)b, hi = (unsigned)(b >> 32);
    if constexpr (O == 8) {  // row_ror:8 swaps the two halves of each 16-lane row
        const unsigned rlo = (unsigned)__builtin_amdgcn_update_dpp(0, (int)lo, 0x128, 0xF, 0xF, false);
        const unsigned rhi = (unsigned)__builtin_amdgcn_update_dpp(0, (int)hi, 0x128, 0xF, 0xF, false);
        return x + __longlong_as_double(((unsigned long long)rhi << 32) | rlo);
    } else {
        // permlane swaps pair rows (16) or wave halves (32); both outputs hold
        // the lower lane's value first, so the sum is the same on both lanes
        const auto L = O == 16 ? __builtin_amdgcn_permlane16_swap(lo, lo, false, false)
                               : __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
        const auto Hi = O == 16 ? __builtin_amdgcn_permlane16_swap(hi, hi, false, false)
                                : __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
        const double a = __longlong_as_double(((unsigned long long)Hi[0] << 32) | L[0]);
        const double c = __longlong_as_double(((unsigned long long)Hi[1] << 32) | L[1]);
        return a + c;
    }
}

// Column sums of per-lane fp64 partials (each lane holds EPL columns of its
// chunk), in a fixed order: thread t < D receives the total of column t (no
// other thread receives anything).  `red` holds NW*D doubles; the caller
// orders any later reuse of it with a barrier of its own.
// One step of a halving sum over the lane pairs (l, l ^ O), O = 16 or 32:
// the lower lane of each pair keeps p, the upper one q, each summed over the
// pair with the lower lane's value first (as xor_sum adds).
template <int O> __device__ __forceinline__ double pair_sum_split(double p, double q) {
    const unsigned long long bp = __double_as_longlong(p), bq = __double_as_longlong(q);
    const unsigned plo = (unsigned)bp, phi = (unsigned)(bp >> 32), qlo = (unsigned)bq, qhi = (unsigned)(bq >> 32);
    const auto L = O == 16 ? __builtin_amdgcn_permlane16_swap(plo, qlo, false, false)
                           : __builtin_amdgcn_permlane32_swap(plo, qlo, false, false);
    const auto H = O == 16 ? __builtin_amdgcn_permlane16_swap(phi, qhi, false, false)
                           : __builtin_amdgcn_permlane32_swap(phi, qhi, false, false);
    return __longlong_as_double(((unsigned long long)H[0] << 32) | L[0]) +
           __longlong_as_double(((unsigned long long)H[1] << 32) | L[1]);
}
template <int DT, int D>
__device__ __forceinline__ double block_col_total(double *acc, double *red, int red_cap) {
    using S = Shape<DT, D>;
    constexpr int E = S::EPL;
    // The wave's row groups are summed in halving steps (lanes 16 apart, then
    // 32 apart), each lane keeping half of its columns per step, in the same
    // association and operand order as summing each column over the row
    // groups; each lane then writes the totals of the columns it kept.
    if constexpr (S::LPR <= 8) {
#pragma unroll
        for (int i = 0; i < E; ++i) acc[i] = xor_sum<8>(acc[i]);
    }
    const int lane = lane_id(), w = wave_id();
    constexpr int M16 = S::LPR <= 16 ? E / 2 : E;      // columns kept after the step over lanes 16 apart
    constexpr int M32 = S::LPR <= 32 ? M16 / 2 : M16;  // and after the one over lanes 32 apart
    static_assert(M32 >= 1, "at least one column per lane");
    int first = 0;  // the first of this lane's columns within its E
    double v16[M16], v32[M32];
#pragma unroll
    for (int i = 0; i < M16; ++i) v16[i] = S::LPR <= 16 ? pair_sum_split<16>(acc[i], acc[i + M16 % E]) : acc[i];
    if constexpr (S::LPR <= 16) first += ((lane >> 4) & 1) * M16;
#pragma unroll
    for (int i = 0; i < M32; ++i) v32[i] = S::LPR <= 32 ? pair_sum_split<32>(v16[i], v16[(i + M32) % M16]) : v16[i];
    if constexpr (S::LPR <= 32) first += (lane >> 5) * M32;
    if (S::LPR > 8 || (lane & 8) == 0)  // lanes 8 apart hold the same totals
#pragma unroll
        for (int i = 0; i < M32; ++i) red[lds_ix<kSiteRed>(w * D + (lane % S::LPR) * E + first + i, red_cap)] = v32[i];
    __syncthreads();
    static_assert(D <= NT, "one thread per column");
    double s = 0.0;
    if (threadIdx.x < D) {
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) s += red[lds_ix<kSiteRed>(ww * D + threadIdx.x, red_cap)];
    }
    return s;
}

// ---------------------------------------------------------------- selection

// The wave index as a scalar (the compiler cannot prove threadIdx.x / 64
// uniform, and per-wave loops and offsets would otherwise run on vector
// registers under exec masks).
__device__ __forceinline__ int wave_id_s() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Number of set bits of a ballot mask in the lanes below this one.
__device__ __forceinline__ uint32_t ballot_rank(uint64_t m) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Sum of x over lanes 0..i-1 (i uniform, 0 <= i <= 16) of a value held by lanes 0..15.
__device__ __forceinline__ uint32_t sum_below16(uint32_t x, int i) {
    const uint32_t incl = wave_incl_scan(x);
    return i > 0 ? lane_u32(incl, i - 1) : 0u;
}

// Threshold and lists for the fused pass.  The kept set is the first N
// elements in (key desc, slot asc) order; with (T, J) the N-th of them,
// keep(j) <=> key_j > T or (key_j == T and j <= J).
//
// Before the barrier that ended scoring every wave has stored its key minimum
// in bc[w] and maximum in bc[16 + w], and hist[] and the candidate counter
// bc[100] are zero; hist2[] (kBins entries, just past the keys) is
// scratch.  Wave w owns the slots [j0, j1): a run of whole 64-slot blocks,
// one more block for the first (blocks mod NW) waves, so that the four waves
// of each SIMD (w, w+4, w+8, w+12) hold equal shares to within one block (a
// sweep ends when the busiest SIMD has issued its waves' blocks).
// Histogram passes over the key range narrow it to one bin (the two histogram
// buffers alternate, so a pass costs two barriers).  Once the bin holds at
// most kCand keys, one sweep gathers them and publishes every wave's counts of
// the sure evictions (below the bin) and sure movers (above it); the waves
// rank the candidates between them to find (T, J), after which every wave
// knows the decision on every candidate and hence its own list offsets
// without a further count.  If the bin holds more than kCand keys they are
// all equal and J is found by counting equal keys in slot order.  evl
// receives every evicted slot and mvl every kept slot >= N, both ascending (so
// evl starts with the holes below N); keep_out is written if given.  Returns
// the number of movers.
// keys_words: 32-bit words of the keys region (the keys, then hist2).
// Touches (the fused pass): the sweep that gathers the candidates also reads
// one word of each 128-byte line (at most kTouchLines per row) of the V row of
// every slot below N that surely leaves or is a candidate (a hole, whose V row
// the gather reads for the running sum) and of the K row of every slot at or
// above N that surely stays or is a candidate (a mover) (tv, tk: the unit's V
// and K, ss: bytes per slot; null: no touch), so that the gather finds those
// rows in L2.  The words land in tch, which the caller
// keeps live until the gather is done (a register reused earlier would make
// the wave wait for its load); only the sweep's first kTouchIters blocks of 64
// slots touch.
constexpr int kTouchIters = 4, kTouchLines = 2;
__device__ __forceinline__ int select_and_build(const uint32_t *keys, int n, int N, uint32_t *evl, int evict_cap,
                                                uint32_t *mvl, int move_cap, uint8_t *keep_out, LdsHead &H,
                                                int keys_words, const char *tv, const char *tk, uint32_t ss,
                                                int row_bytes, uint32_t (&tch)[kTouchIters][kTouchLines]) {
    uint32_t *const hist2 = const_cast<uint32_t *>(keys) + ((n + 3) & ~3);
    const int hist2_cap = keys_words - ((n + 3) & ~3);
    const int w = wave_id_s(), lane = lane_id();
    const int blocks = (n + 63) >> 6, per = blocks / NW, extra = blocks % NW;
    const int j0 = 64 * (w * per + min(w, extra));
    const int j1 = min(n, j0 + 64 * (per + (w < extra ? 1 : 0)));
    uint32_t lo = wave_min_u32(lane < NW ? H.bc[lane] : 0xFFFFFFFFu);
    uint32_t hi = wave_max_u32(lane < NW ? H.bc[16 + lane] : 0u);
    int need = N;       // 1-based rank of (T, J) among the keys in [lo, hi]
    int in_range = n;   // keys in [lo, hi]
    // The bin of histogram hc (bins in descending key order, wave w owning
    // bins kBins-1-64w .. kBins-64-64w) that holds the need-th largest key:
    // its index, its count and the count of the keys above it; the other
    // buffer hn is cleared on the way (it was last read before the barrier
    // that precedes the call).
    struct Bin { int b; uint32_t h, above; };
    auto find_bin = [&](const uint32_t *hc, int hc_cap, uint32_t *hn, int hn_cap)
                        __attribute__((always_inline)) -> Bin {
        const uint32_t total = wave_incl_scan(hc[lds_ix<kSiteHist>(kBins - 1 - threadIdx.x, hc_cap)]);
        hn[lds_ix<kSiteHist>(threadIdx.x, hn_cap)] = 0u;  // NT == kBins
        if (lane == 63) H.bc[80 + w] = total;
        __syncthreads();
        const uint32_t un = (uint32_t)need;
        const uint32_t wt = lane < NW ? H.bc[80 + lane] : 0u;
        const uint32_t wincl = wave_incl_scan(wt);
        // the wave holding it (the totals sum to in_range >= need, so one lane qualifies)
        const int tw = max(__ffsll(__ballot(lane < NW && wincl >= un)) - 1, 0);
        const uint32_t before = lane_u32(wincl - wt, tw);
        const uint32_t hb = hc[lds_ix<kSiteHist>(kBins - 1 - (tw * 64 + lane), hc_cap)];
        const uint32_t bincl = wave_incl_scan(hb) + before;
        const int tl = max(__ffsll(__ballot(bincl >= un)) - 1, 0);
        const uint32_t h = lane_u32(hb, tl);
        return Bin{kBins - 1 - (tw * 64 + tl), h, lane_u32(bincl, tl) - h};
    };
    for (int pass = 0; in_range > kCand && lo != hi; ++pass) {
        uint32_t *hc = (pass & 1) ? hist2 : H.hist;
        uint32_t *hn = (pass & 1) ? H.hist : hist2;
        const int hc_cap = (pass & 1) ? hist2_cap : kBins;
        const int hn_cap = (pass & 1) ? kBins : hist2_cap;
        const int bits = 32 - __clz(hi - lo);  // bits of the largest offset
        const int shift = bits > 10 ? bits - 10 : 0;
        // a lane outside the range adds 0 to a bin of its own (no lane mask switched)
        for (int jb = j0; jb < j1; jb += 64) {
            const int j = jb + lane;
            const uint32_t k = keys[lds_ix<kSiteKeys>(j < j1 ? j : j0, n)];
            const bool in = j < j1 && k >= lo && k <= hi;
            atomicAdd(&hc[lds_ix<kSiteHist>(in ? (int)((k - lo) >> shift) : lane, hc_cap)], in ? 1u : 0u);
        }
        __syncthreads();
        const Bin r = find_bin(hc, hc_cap, hn, hn_cap);
        const uint64_t b = (uint64_t)r.b;
        need -= (int)r.above;
        in_range = (int)r.h;
        const uint64_t top = (uint64_t)lo + ((b + 1) << shift) - 1u;
        hi = top < (uint64_t)hi ? (uint32_t)top : hi;
        lo = lo + (uint32_t)(b << shift);
    }
    uint32_t T, J, ev_off, mv_off, mv_tot;
    if (in_range <= kCand) {
        // gather the keys in [lo, hi] and publish this wave's sure evictions
        // (below lo) and sure movers (above hi)
        uint32_t sev = 0u, smv = 0u;
        auto sweep = [&](int jb, auto touchc, uint32_t (&t)[kTouchLines]) __attribute__((always_inline)) {
            const int j = jb + lane;
            const bool v = j < j1;
            const uint32_t k = keys[lds_ix<kSiteKeys>(v ? j : j0, n)];
            const bool c = v && k >= lo && k <= hi;
            const bool gone = v && k < lo, moves = v && k > hi && j >= N;
            sev += __popcll(__ballot(gone));
            smv += __popcll(__ballot(moves));
            if constexpr (decltype(touchc)::value) {
                // (a candidate's row is touched too: half of them leave or move)
                const bool hole = (gone || c) && j < N;
                if (hole || ((moves || (c && j >= N)) && tk)) {
                    // (a two-way select of the base: a three-way one with a null
                    // became a table in scratch memory)
                    const char *row = (hole ? tv : tk) + (uint64_t)j * ss;
#pragma unroll
                    for (int l = 0; l < kTouchLines; ++l)
                        if (l * 128 < row_bytes) t[l] = *reinterpret_cast<const uint32_t *>(row + l * 128);
                }
            }
            const uint64_t m = __ballot(c);
            if (m) {
                uint32_t base = 0u;
                if (lane == 0) base = atomicAdd(&H.bc[100], (uint32_t)__popcll(m));
                base = __builtin_amdgcn_readfirstlane(base);
                const uint32_t slot = base + ballot_rank(m);
                if (c && slot < (uint32_t)kCand) {  // the bin holds exactly in_range <= kCand keys
                    H.cand_key[slot] = k;
                    H.cand_idx[slot] = (uint32_t)j;
                }
            }
        };
        int jb = j0;
        if (tv) {
#pragma unroll
            for (int i = 0; i < kTouchIters; ++i, jb += 64)
                if (jb < j1) sweep(jb, BoolC<true>{}, tch[i]);
        }
        for (; jb < j1; jb += 64) sweep(jb, BoolC<false>{}, tch[0]);
        if (lane == 0) {
            H.bc[32 + w] = sev;
            H.bc[48 + w] = smv;
        }
        __syncthreads();
        // lane t holds candidate t; wave w ranks candidates w, w+16, w+32, w+48
        const int cnt = in_range;
        const bool live = lane < cnt;
        const uint32_t ck = live ? H.cand_key[lane] : 0u;
        const uint32_t ci = live ? H.cand_idx[lane] : 0u;
        for (int i = w; i < cnt; i += NW) {
            const uint32_t ki = lane_u32(ck, i), ji = lane_u32(ci, i);
            const uint32_t rank = __popcll(__ballot(live && (ck > ki || (ck == ki && ci < ji))));
            if (rank == (uint32_t)(need - 1)) {
                if (lane == 0) {
                    H.bc[67] = ki;
                    H.bc[68] = ji;
                }
            }
        }
        const uint32_t se = lane < NW ? H.bc[32 + lane] : 0u;
        const uint32_t sm = lane < NW ? H.bc[48 + lane] : 0u;
        __syncthreads();
        T = H.bc[67];
        J = H.bc[68];
        // list offsets: the sure counts of the waves before this one, plus the
        // candidates in their segments that go (evicted) or move
        const bool ckeep = live && (ck > T || (ck == T && ci <= J));
        const bool cbefore = live && (int)ci < j0;
        ev_off = sum_below16(se, w) + (uint32_t)__popcll(__ballot(cbefore && !ckeep));
        mv_off = sum_below16(sm, w) + (uint32_t)__popcll(__ballot(cbefore && ckeep && (int)ci >= N));
        mv_tot = sum_below16(sm, NW) + (uint32_t)__popcll(__ballot(ckeep && (int)ci >= N));
    } else {
        // every key in [lo, hi] equals T = lo: J is the slot of the need-th of
        // them in slot order
        T = lo;
        uint32_t ce = 0u;
        for (int jb = j0; jb < j1; jb += 64) {
            const int j = jb + lane;
            ce += __popcll(__ballot(j < j1 && keys[lds_ix<kSiteKeys>(j, n)] == T));
        }
        if (lane == 0) H.bc[32 + w] = ce;
        __syncthreads();
        const uint32_t eq_before = sum_below16(lane < NW ? H.bc[32 + lane] : 0u, w);
        if (eq_before < (uint32_t)need && (uint32_t)need <= eq_before + ce) {
            uint32_t r = eq_before;
            for (int jb = j0; jb < j1; jb += 64) {
                const int j = jb + lane;
                const uint64_t m = __ballot(j < j1 && keys[lds_ix<kSiteKeys>(j, n)] == T);
                const uint32_t c = (uint32_t)__popcll(m);
                if (r + c >= (uint32_t)need) {  // the (need - r)-th set lane of m
                    uint64_t mm = m;
                    for (uint32_t q = 1; q < (uint32_t)need - r; ++q) mm &= mm - 1;
                    if (lane == 0) H.bc[68] = (uint32_t)(jb + __ffsll((unsigned long long)mm) - 1);
                    break;
                }
                r += c;
            }
        }
        __syncthreads();
        J = H.bc[68];
        // counts per wave, then offsets
        uint32_t cev = 0u, cmv = 0u;
        for (int jb = j0; jb < j1; jb += 64) {
            const int j = jb + lane;
            const bool v = j < j1;
            const uint32_t k = v ? keys[lds_ix<kSiteKeys>(j, n)] : 0u;
            const bool keep = v && (k > T || (k == T && (uint32_t)j <= J));
            cev += __popcll(__ballot(v && !keep));
            cmv += __popcll(__ballot(keep && j >= N));
        }
        if (lane == 0) {
            H.bc[32 + w] = cev;  // every wave has read bc[32..47] before the barrier above
            H.bc[48 + w] = cmv;
        }
        __syncthreads();
        const uint32_t e_i = lane < NW ? H.bc[32 + lane] : 0u;
        const uint32_t m_i = lane < NW ? H.bc[48 + lane] : 0u;
        ev_off = sum_below16(e_i, w);
        mv_off = sum_below16(m_i, w);
        mv_tot = sum_below16(m_i, NW);
    }
    // each wave writes its part of the lists
    // (a lane with nothing to list stores to its own word of the histogram,
    // which nothing reads any more, so that no lane mask is switched)
    for (int jb = j0; jb < j1; jb += 64) {
        const int j = jb + lane;
        const bool v = j < j1;
        const uint32_t k = keys[lds_ix<kSiteKeys>(v ? j : j0, n)];
        const bool keep = v && (k > T || (k == T && (uint32_t)j <= J));
        const bool ev = v && !keep;
        const bool mv = keep && j >= N;
        const uint64_t mev = __ballot(ev), mmv = __ballot(mv);
        const uint32_t rev = ev_off + ballot_rank(mev);
        const uint32_t rmv = mv_off + ballot_rank(mmv);
        *((ev && rev < (uint32_t)evict_cap) ? evl + lds_ix<kSiteEvl>((int)rev, evict_cap) : H.hist + lane) =
            (uint32_t)j;
        *((mv && rmv < (uint32_t)move_cap) ? mvl + lds_ix<kSiteMvl>((int)rmv, move_cap) : H.hist + 64 + lane) =
            (uint32_t)j;
        if (keep_out && v) keep_out[j] = keep ? 1 : 0;
        ev_off += (uint32_t)__popcll(mev);
        mv_off += (uint32_t)__popcll(mmv);
    }
    __syncthreads();
    return (int)mv_tot;
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
    const int keys_words = (p.off_lists - p.off_keys) / 4;  // the keys region (keys, hist2; red)
    const int red_cap = (p.off_lists - p.off_keys) / 8;

    const int head = blockIdx.x, layer = blockIdx.y, sl = blockIdx.z;
    const int ul = (sl * p.num_layers + layer) * p.num_kv_heads + head;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl], N = p.nN[2 * sl + 1];
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    const char *vb = p.v + off;
    const uint32_t ss32 = p.s_slot;
    const int64_t cap = p.capacity;
    const int lane = lane_id();
    const int cl = lane % S::LPR;

    // Every argument needed before the first row load is fetched here, in one
    // batch of scalar loads (the empty asm keeps the compiler from spreading
    // the loads over the branches below, one round trip each).
    double *const arg_rs = p.running_sum;
    float *const arg_scores = p.scores;
    uint8_t *const arg_keep = p.keep;
    const int arg_mode = p.mode, arg_stash = p.stash_rows;
    asm volatile("" ::"s"(arg_rs), "s"(arg_scores), "s"(arg_keep), "s"(arg_mode), "s"(arg_stash), "s"(n),
                 "s"(N), "s"(vb), "s"(ss32));
    const bool score_mode = arg_mode == kModeScore;
    double *st = arg_rs ? arg_rs + u * (D + 1) : nullptr;  // null in kModeScore
    const bool evict = !score_mode && n > N;
    float *scores_out = arg_scores ? arg_scores + u * cap : nullptr;
    uint8_t *keep_out = arg_keep ? arg_keep + u * cap : nullptr;

    const bool need_scores = score_mode || evict || scores_out;

    // The rows are read in one software-pipelined stream of tiles over two
    // parts: first the rows not yet in the running sum, [count, n), which give
    // the mean (staged in LDS as far as they fit), then the rows still to be
    // scored: [0, count) and the first part's unstaged rows.  The state's
    // token count and column sums are read first.  The
    // first tile goes out right behind them for the steady-state guess
    // count = min(N, n) and goes out again only if the guess was wrong, so that
    // either way exactly one tile is in flight, in the same order, and every
    // wait counts exactly.  Nothing branches before these loads (a unit with
    // no rows reads row 0 of its slab and ignores it): the kernel arguments
    // arrive in one batch and the row tiles go out right behind them.
    const double *stp = st ? st : reinterpret_cast<const double *>(vb);
    const double craw = stp[st ? D : 0];
    const double st_col = stp[st ? min((int)threadIdx.x, D) : 0];
    const int lastrow = max(n - 1, 0);
    constexpr int kStep = S::GROUPS * kChunks;  // rows per tile of the stream
    // A first part of at most one row per lane group (a decode step appends
    // one row) is read by a single chunk issued ahead of the first tile, so
    // that the stream starts with rows to score instead of a tile of repeats.
    // The first part is staged in LDS as far as it fits (its first `staged`
    // rows); the scoring part then covers the old rows and the rest of the
    // first part: element e of it is row e below cnt and row e + staged above.
    struct Plan {
        int cnt, fresh, staged, tiles_f, second, tiles;  // second: rows of the scoring part
        bool small;                                      // first part in one chunk, staged
    };
    auto plan_for = [&](int cnt) __attribute__((always_inline)) {
        Plan q;
        q.cnt = cnt;
        q.fresh = n - cnt;
        q.staged = min(q.fresh, arg_stash);
        q.small = q.fresh > 0 && q.fresh <= S::GROUPS && q.fresh <= arg_stash;
        q.tiles_f = q.small ? 0 : (q.fresh + kStep - 1) / kStep;
        q.second = !need_scores ? 0 : n - q.staged;
        q.tiles = q.tiles_f + (q.second + kStep - 1) / kStep;
        return q;
    };
    auto srow = [&](const Plan &q, int e) __attribute__((always_inline)) { return e < q.cnt ? e : e + q.staged; };
    // chunk k of tile t of the stream; a tile past the end reads the last row
    // (never used)
    auto load_chunk = [&](const Plan &q, int t, int k, uint32_t z = 0u) __attribute__((always_inline)) -> uint4 {
        const bool first = t < q.tiles_f;
        const int lim = first ? q.fresh : q.second;
        const int rbase = first ? q.cnt : 0;
        const int e = (first ? t : t - q.tiles_f) * kStep + (k * NW + wave_id()) * S::RPW + lane / S::LPR;
        const int ec = min(e, lim - 1);
        const int r = (t < q.tiles && lim > 0) ? (first ? rbase + ec : srow(q, ec)) : lastrow;
        return load_stream(vb, row_off(r, ss32, cl) + z);
    };
    auto load_v = [&](const Plan &q, int t, uint4 (&buf)[kChunks]) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < kChunks; ++k) buf[k] = load_chunk(q, t, k);
    };
    const int eb = wave_id() * S::RPW + lane / S::LPR;  // this lane's row group
    auto load_small = [&](const Plan &q) __attribute__((always_inline)) -> uint4 {
        return load_stream(vb, row_off(min(q.cnt + eb, lastrow), ss32, cl));
    };
    const Plan guessed = plan_for(st ? min(N, n) : 0);
    uint4 buf[kChunks], fc;
    if (guessed.small) fc = load_small(guessed);
    load_v(guessed, 0, buf);

    if (n <= 0) {
        if (st) {
            for (int t = threadIdx.x; t <= D; t += NT) st[t] = 0.0;
        }
        return;
    }
    if (!need_scores && !st) {
        for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = 1;
        return;
    }
    int count = 0;
    if (st) count = (craw >= 0.0 && craw <= (double)n && craw == (double)(int)craw) ? (int)craw : 0;
    const Plan q = count == guessed.cnt ? guessed : plan_for(count);
    if (count != guessed.cnt) {
        if (q.small) fc = load_small(q);
        load_v(q, 0, buf);
    }
    const int fresh = q.fresh;
    const int staged = q.staged;             // first-part rows in LDS
    const bool stashed = staged == fresh;    // all of them
    auto sfetch = [&](int r, int c) __attribute__((always_inline)) -> uint4 {
        return *reinterpret_cast<const uint4 *>(stash + (int64_t)lds_ix<kSiteStash>(r - count, p.stash_rows) * S::ROWB +
                                                c * 16);
    };
    auto fresh_row = [&](int e) __attribute__((always_inline)) { return count + min(e, max(staged - 1, 0)); };
    const bool amode = evict && n == N + 1;  // decode: exactly one token goes
    // keys go to LDS for the selection and for the score output: no global
    // store sits between the row loads of the stream (a store in flight makes
    // every later load wait for all outstanding memory operations)
    const bool to_lds = evict || scores_out;
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;   // this thread's key range
    float m[S::EPL];                          // this lane's columns of v_bar (Dir: v_bar / |v_bar|)
    float ml[S::EPL];                         // L2: their low parts (v_bar - m, rounded)
    bool mean_zero = false;

    // ---- mean: sum the rows not yet summed (Sec. 3.2, Eq. vd) ----
    double acc[S::EPL];
#pragma unroll
    for (int i = 0; i < S::EPL; ++i) acc[i] = 0.0;
    auto mean_body = [&](int e, bool valid, uint4 w) __attribute__((always_inline)) {
        float x[S::EPL];
        E::unpack(w, x);
        if (valid) {
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) acc[i] += (double)x[i];
            if (e < staged)
                *reinterpret_cast<uint4 *>(stash + (int64_t)lds_ix<kSiteStash>(e, p.stash_rows) * S::ROWB + cl * 16) = w;
        }
    };
    auto finish_mean = [&]() __attribute__((always_inline)) {
        const double fresh_sum = block_col_total<DT, D>(acc, red, red_cap);
        if (threadIdx.x < D) {
            const int t = threadIdx.x;
            const double old_sum = count > 0 ? st_col : 0.0;
            const double s = old_sum + fresh_sum;
            H.old_sum[t] = old_sum;
            H.sum[t] = s;
            const double mean = s / (double)n;
            const float hi = (float)mean;
            H.mean[t] = hi;
            if constexpr (VAR == kL2) H.aux[t] = (float)(mean - (double)hi);
        }
        __syncthreads();
        if constexpr (VAR == kDir) {
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
            for (int t = threadIdx.x; t < D; t += NT) H.aux[t] = mean_zero ? 0.f : H.mean[t] / mn;
            __syncthreads();
        }
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) {
            m[i] = (VAR == kDir ? H.aux : H.mean)[cl * S::EPL + i];
            ml[i] = VAR == kL2 ? H.aux[cl * S::EPL + i] : 0.f;
        }
    };

    // ---- scores (Sec. 3.2) ----
    auto on_row = [&](int r, bool valid, uint4 w) __attribute__((always_inline)) -> float {
        float x[S::EPL];
        E::unpack(w, x);
        float s;
        if constexpr (VAR == kL2) {  // L2: ||v - v_bar||, v_bar as a pair m + ml of fp32
                                   // numbers, so that the difference keeps fp32
                                   // accuracy however far v_bar lies from the origin
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) {
                const float t = (x[i] - m[i]) - ml[i];
                a = fmaf(t, t, a);
            }
            s = score_sqrt(row_sum<S::LPR>(a));
        } else if constexpr (VAR == kNorm || VAR == kKeepSmallest) {  // Norm: ||v||
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) a = fmaf(x[i], x[i], a);
            s = score_sqrt(row_sum<S::LPR>(a));
        } else {  // Dir: 1 - cos = ||v/|v| - v_bar/|v_bar| ||^2 / 2
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) a = fmaf(x[i], x[i], a);
            const float nv2 = row_sum<S::LPR>(a);
            const bool ok = nv2 > 0.f && !mean_zero;
            const float inv = ok ? score_rsqrt(nv2) : 0.f;
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
            const uint32_t key = key_of<VAR>(s);
            if (to_lds) {
                keys[lds_ix<kSiteKeys>(r, p.keys_cap)] = key;
                kmin = min(kmin, key);
                kmax = max(kmax, key);
            }
        }
        return s;
    };

    auto on_fresh = [&](int e, bool valid, uint4 w) __attribute__((always_inline)) { on_row(count + e, valid, w); };
    // L2 and Norm score the four chunks of a tile together (one square root per
    // lane, one key store per row); chunk k of the tile holds element
    // e0 + k*NW*RPW of this lane's row group, valid below lim, at row rbase + e
    constexpr bool kBatch = VAR != kDir && kUnroll == 4 && kChunks % 4 == 0;
    auto partial = [&](uint4 w) __attribute__((always_inline)) {
        float x[S::EPL];
        E::unpack(w, x);
        float a = 0.f;
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) {
            const float t = VAR == kL2 ? (x[i] - m[i]) - ml[i] : x[i];
            a = fmaf(t, t, a);
        }
        return a;
    };
    // (the row of element e is rbase + e, plus gap at and above gap_at)
    auto score4 = [&](const float (&a)[4], int e0, int lim, int rbase, int gap_at, int gap) __attribute__((always_inline)) {
        const float s = score_sqrt(row_sums4<S::LPR>(a, cl));
        const int e = e0 + quad_row(cl) * NW * S::RPW;
        if (cl < 4 && e < lim) {
            const uint32_t key = key_of<VAR>(s);
            if (to_lds) {
                keys[lds_ix<kSiteKeys>(rbase + e + (e >= gap_at ? gap : 0), p.keys_cap)] = key;
                kmin = min(kmin, key);
                kmax = max(kmax, key);
            }
        }
    };
    // staged tile i (rows count + [i*STEP, (i+1)*STEP)) scored from LDS
    auto score_stash_tile = [&](int i) __attribute__((always_inline)) {
        const int e0 = i * S::STEP + wave_id() * S::RPW + lane / S::LPR;
        if constexpr (kBatch) {
            uint4 w4[kUnroll];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) w4[k] = sfetch(fresh_row(e0 + k * NW * S::RPW), cl);
            float a[4];
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) a[k] = partial(w4[k]);
            score4(a, e0, staged, count, staged, 0);
        } else {
#pragma unroll
            for (int k = 0; k < kUnroll; ++k) {
                const int e = e0 + k * NW * S::RPW;
                on_fresh(e, e < staged, sfetch(fresh_row(e), cl));
            }
        }
    };
    const bool score_stash = staged > 0 && need_scores;
    const int stash_tiles = score_stash ? (staged + S::STEP - 1) / S::STEP : 0;
    // Tile t is used chunk by chunk, and chunk k of tile t + 1 is requested
    // into the same registers as soon as chunk k of t is used: the row loads
    // in flight never drop below one tile less one chunk, and the loads cross
    // from the first part to the second unbroken (the first scoring tile is in
    // flight while the mean is finished).  The two parts run as two loops, so
    // that the mean's fp64 partials are dead while the scoring part runs.  The
    // staged rows are scored from LDS one tile after each scoring tile but the
    // last, while the next tile's rows are on their way (scored at the switch
    // they would keep the wave from issuing loads for a while, with one tile
    // in flight), and any left after the last but one.
    // chunk k of scoring tile tn < tiles (no clamping to other parts needed)
    auto load_scored = [&](int tn, int k, uint32_t z) __attribute__((always_inline)) -> uint4 {
        const int e = (tn - q.tiles_f) * kStep + k * NW * S::RPW + eb;
        return load_stream(vb, row_off(srow(q, min(e, q.second - 1)), ss32, cl) + z);
    };
    // The load that refills a chunk's registers takes its address through a
    // zero that the compiler sees as computed from the chunk's results, so it
    // is issued after the chunk's last use (issued earlier, it would land in
    // other registers, copied back at the loop's end, which waits for it),
    // and no later work moves above it (the loads stay spread out, so that
    // about one tile stays in flight).
    auto use_fresh = [&](int t, auto more) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < kChunks; ++k) {
            const int e = t * kStep + k * NW * S::RPW + eb;
            mean_body(e, e < fresh, buf[k]);
            if constexpr (more()) {
                buf[k] = load_chunk(q, t + 1, k, zero_after(acc));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    auto use_scored = [&](int t, auto more) __attribute__((always_inline)) {
        const int e0 = (t - q.tiles_f) * kStep + eb;
        if constexpr (kBatch) {
#pragma unroll
            for (int h = 0; h < kChunks; h += 4) {
                float a[4];
#pragma unroll
                for (int k = h; k < h + 4; ++k) {
                    a[k - h] = partial(buf[k]);
                    if constexpr (more()) {
                        buf[k] = load_scored(t + 1, k, zero_after(a[k - h]));
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
                score4(a, e0 + h * NW * S::RPW, q.second, 0, q.cnt, q.staged);
            }
        } else {
#pragma unroll
            for (int k = 0; k < kChunks; ++k) {
                const int e = e0 + k * NW * S::RPW;
                const float sc = on_row(srow(q, e), e < q.second, buf[k]);
                if constexpr (more()) {
                    buf[k] = load_scored(t + 1, k, zero_after(sc));
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };
    {
        const int T = q.tiles;
        int t = 0;
        if (q.small) mean_body(eb, eb < fresh, fc);
        for (; t < q.tiles_f && t + 1 < T; ++t) use_fresh(t, std::true_type{});
        if (t < q.tiles_f) use_fresh(t++, std::false_type{});  // no scoring part follows
        finish_mean();
        int si = 0;  // staged tiles scored
        for (; t + 1 < T; ++t) {
            use_scored(t, std::true_type{});
            if (si < stash_tiles) score_stash_tile(si++);
        }
        for (; si < stash_tiles; ++si) score_stash_tile(si);
        if (t < T) use_scored(t, std::false_type{});  // the last tile: no load past the end
    }
    if (to_lds) {  // what the selection reads after the barrier below
        kmin = wave_min_u32(kmin);
        kmax = wave_max_u32(kmax);
        if (lane == 0) {
            H.bc[wave_id()] = kmin;
            H.bc[16 + wave_id()] = kmax;
        }
        H.hist[threadIdx.x] = 0u;  // NT == kBins
        if (threadIdx.x == 0) H.bc[100] = 0u;  // candidate count
    }
    __syncthreads();
    // Every row load of the stream has been used by now.  Saying so keeps the
    // compiler from waiting, at a later reuse of a stream register, for loads
    // it cannot prove complete, which would then include the selection's touches.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    if (scores_out)  // the key holds the score's bits
        for (int j = threadIdx.x; j < n; j += NT) scores_out[j] = score_of<VAR>(keys[lds_ix<kSiteKeys>(j, p.keys_cap)]);
    if (score_mode) {  // the mean leaves after the stream, like the scores
        if (p.mean_out)
            for (int t = threadIdx.x; t < D; t += NT) p.mean_out[u * D + t] = H.mean[t];
        return;
    }

    // ---- select (Sec. 2.1, Eq. eviction) ----
    int n_moves = 0;
    uint32_t tch[kTouchIters][kTouchLines] = {};  // rows the selection fetched into L2 for the gather
    if (evict) {
        if (amode) {
            // (key << 32) | ~slot: the minimum is the lowest score, highest slot
            uint64_t best = ~0ull;
            for (int j = threadIdx.x; j < n; j += NT) {
                const uint64_t c = ((uint64_t)keys[lds_ix<kSiteKeys>(j, p.keys_cap)] << 32) |
                                   (uint64_t)(0xFFFFFFFFu - (uint32_t)j);
                best = c < best ? c : best;
            }
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
                evl[lds_ix<kSiteEvl>(0, p.evict_cap)] = (uint32_t)victim;
                mvl[lds_ix<kSiteMvl>(0, p.move_cap)] = (uint32_t)N;  // slot N = n - 1 is kept unless it is the victim
            }
            n_moves = victim < N ? 1 : 0;
            for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = j == victim ? 0 : 1;
            __syncthreads();
        } else {
            (void)lds_ix<kSiteKeys>(n - 1, p.keys_cap);  // the keys fit their region
            n_moves = select_and_build(keys, n, N, evl, p.evict_cap, mvl, p.move_cap, keep_out, H,
                                       keys_words, vb, p.k ? p.k + off : nullptr, ss32, S::ROWB, tch);
        }
    } else {
        for (int j = threadIdx.x; keep_out && j < n; j += NT) keep_out[j] = 1;
    }

    // ---- gather with slot reuse, and the evicted rows leave the running sum ----
    // In steady state (the state covered exactly the N old rows) the new sum is
    // old - holes + movers, so only the rows that move are read; otherwise it
    // is total - every evicted row.
    if (evict) {
        const int n_ev = n - N;  // evl[0, n_moves) are the holes, the rest lie at or above N
        const bool steady = st && count == N;
        char *kb = p.k ? p.k + off : nullptr;
        char *vw = p.v + off;
        int32_t *pos = p.pos ? p.pos + u * cap : nullptr;
        const int g = wave_id() * S::RPW + lane / S::LPR;  // row group of this lane
        auto vfetch = [&](int r) __attribute__((always_inline)) -> uint4 {
            return (r >= count && r < count + staged) ? sfetch(r, cl) : load_stream(vb, row_off(r, ss32, cl));
        };
        double acc[S::EPL];
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) acc[i] = 0.0;
        if (!st || steady) {
            // Only the moved rows are touched.  A wave takes only the slots of a
            // batch that hold a moved row for it, so no load is spent on padding;
            // the list reads come first, then every row load of the batch, then
            // the stores, with no load waiting behind another.
            const char *ksrc = kb ? kb : vb;  // without K a V row stands in, unused
            const int wrow = wave_id() * S::RPW;
            auto batch = [&](int e0, auto kvc, auto stashc) __attribute__((always_inline)) {
                constexpr int KV = decltype(kvc)::value;
                constexpr bool STASH = decltype(stashc)::value;
                int dst[KV], src[KV];
#pragma unroll
                for (int k = 0; k < KV; ++k) {
                    const int e = e0 + k * S::GROUPS + g;
                    const int ec = e < n_moves ? e : n_moves - 1;
                    dst[k] = (int)evl[lds_ix<kSiteEvl>(ec, p.evict_cap)];
                    src[k] = (int)mvl[lds_ix<kSiteMvl>(ec, p.move_cap)];
                }
                uint4 vh[KV], km[KV], vm[KV];
                int32_t ps[KV];
                // Row loads in the order their data is needed: the moved K and V
                // rows feed the stores, the hole rows only the running sum.  They
                // are non-temporal (scattered rows read once gain nothing from L2
                // allocation and, measured, move markedly slower with it), and all
                // are unconditional (without a state a hole row is read and
                // ignored) so that no use can be hoisted next to its load.
#pragma unroll
                for (int k = 0; k < KV; ++k)
                    km[k] = load_stream(ksrc, row_off(src[k], ss32, cl));
                if constexpr (!STASH) {  // staged movers (a partly staged block) come from LDS
#pragma unroll
                    for (int k = 0; k < KV; ++k)
                        vm[k] = src[k] < count + staged ? sfetch(src[k], cl)
                                                        : load_stream(vb, row_off(src[k], ss32, cl));
                }
                if (pos) {
#pragma unroll
                    for (int k = 0; k < KV; ++k) ps[k] = pos[src[k]];
                }
#pragma unroll
                for (int k = 0; k < KV; ++k) vh[k] = load_stream(vb, row_off(dst[k], ss32, cl));
                if constexpr (STASH) {
#pragma unroll
                    for (int k = 0; k < KV; ++k) vm[k] = sfetch(src[k], cl);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int k = 0; k < KV; ++k) {
                    const int e = e0 + k * S::GROUPS + g;
                    if (e >= n_moves) continue;
                    if (kb) store_stream(kb, row_off(dst[k], ss32, cl), km[k]);
                    store_stream(vw, row_off(dst[k], ss32, cl), vm[k]);
                    if (pos && cl == 0) pos[dst[k]] = ps[k];
                }
                if (st) {  // new sum = old - holes + movers
#pragma unroll
                    for (int k = 0; k < KV; ++k) {
                        const int e = e0 + k * S::GROUPS + g;
                        if (e >= n_moves) continue;
                        float x[S::EPL], y[S::EPL];
                        E::unpack(vh[k], x);
                        E::unpack(vm[k], y);
#pragma unroll
                        for (int i = 0; i < S::EPL; ++i) acc[i] += (double)y[i] - (double)x[i];
                    }
                }
            };
            static_assert(kUnroll == 4, "the batch dispatch below covers 1..4 slots");
            using I1 = IntC<1>;
            using I2 = IntC<2>;
            using I3 = IntC<3>;
            using I4 = IntC<4>;
            for (int e0 = 0; e0 < n_moves; e0 += S::STEP) {
                const int left = n_moves - e0 - wrow;  // slot k holds a row for this wave iff k*GROUPS < left
                const int kv = left <= 0 ? 0 : min(kUnroll, (left + S::GROUPS - 1) / S::GROUPS);
                if (stashed) {
                    if (kv == 4) batch(e0, I4{}, BoolC<true>{});
                    else if (kv == 3) batch(e0, I3{}, BoolC<true>{});
                    else if (kv == 2) batch(e0, I2{}, BoolC<true>{});
                    else if (kv == 1) batch(e0, I1{}, BoolC<true>{});
                } else {
                    if (kv == 4) batch(e0, I4{}, BoolC<false>{});
                    else if (kv == 3) batch(e0, I3{}, BoolC<false>{});
                    else if (kv == 2) batch(e0, I2{}, BoolC<false>{});
                    else if (kv == 1) batch(e0, I1{}, BoolC<false>{});
                }
            }
        } else {
            // the state did not cover exactly the N old rows: remove every evicted row
            for (int e0 = 0; e0 < n_ev; e0 += S::STEP) {
                uint4 vh[kUnroll], km[kUnroll], vm[kUnroll];
#pragma unroll
                for (int k = 0; k < kUnroll; ++k) {
                    const int e = e0 + k * S::GROUPS + g;
                    const int ec = e < n_ev ? e : n_ev - 1;
                    vh[k] = vfetch((int)evl[lds_ix<kSiteEvl>(ec, p.evict_cap)]);
                    if (ec < n_moves) {
                        const int src = (int)mvl[lds_ix<kSiteMvl>(ec, p.move_cap)];
                        km[k] = kb ? load_stream(kb, row_off(src, ss32, cl)) : make_uint4(0u, 0u, 0u, 0u);
                        vm[k] = vfetch(src);
                    }
                }
#pragma unroll
                for (int k = 0; k < kUnroll; ++k) {
                    const int e = e0 + k * S::GROUPS + g;
                    if (e >= n_ev) continue;
                    float x[S::EPL];
                    E::unpack(vh[k], x);
#pragma unroll
                    for (int i = 0; i < S::EPL; ++i) acc[i] -= (double)x[i];
                    if (e < n_moves) {
                        const int dst = (int)evl[lds_ix<kSiteEvl>(e, p.evict_cap)];
                        const int src = (int)mvl[lds_ix<kSiteMvl>(e, p.move_cap)];
                        if (kb) store_stream(kb, row_off(dst, ss32, cl), km[k]);
                        store_stream(vw, row_off(dst, ss32, cl), vm[k]);
                        if (pos && cl == 0) pos[dst] = pos[src];
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < kTouchIters; ++i)
#pragma unroll
            for (int l = 0; l < kTouchLines; ++l) asm volatile("" ::"v"(tch[i][l]));
        if (st) {
            const double delta = block_col_total<DT, D>(acc, red, red_cap);  // red aliases keys, no longer needed
            if (threadIdx.x < D) st[threadIdx.x] = (steady ? H.old_sum[threadIdx.x] : H.sum[threadIdx.x]) + delta;
            if (threadIdx.x == 0) st[D] = (double)N;
        }
    } else if (st) {
        for (int t = threadIdx.x; t < D; t += NT) st[t] = H.sum[t];
        if (threadIdx.x == 0) st[D] = (double)n;
    }
}

// Standalone selection: scores (global) -> keep mask.
__global__ void __launch_bounds__(NT) select_kernel(const UnitParams p) {
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    uint32_t *keys = reinterpret_cast<uint32_t *>(lds + p.off_keys);
    const int sl = blockIdx.z;
    const int ul = (sl * p.num_layers + blockIdx.y) * p.num_kv_heads + blockIdx.x;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl], N = p.nN[2 * sl + 1];
    const int64_t cap = p.capacity;
    const float *sc = p.scores_in + u * cap;
    uint8_t *keep = p.keep + u * cap;
    if (n <= N) {
        for (int j = threadIdx.x; j < n; j += NT) keep[j] = 1;
        return;
    }
    uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
    for (int j = threadIdx.x; j < n; j += NT) {
        const uint32_t k = orderable(sc[j]);
        keys[lds_ix<kSiteKeys>(j, p.keys_cap)] = k;
        kmin = min(kmin, k);
        kmax = max(kmax, k);
    }
    kmin = wave_min_u32(kmin);
    kmax = wave_max_u32(kmax);
    if (lane_id() == 0) {
        H.bc[wave_id()] = kmin;
        H.bc[16 + wave_id()] = kmax;
    }
    H.hist[threadIdx.x] = 0u;  // NT == kBins
    if (threadIdx.x == 0) H.bc[100] = 0u;
    __syncthreads();
    uint32_t tch[kTouchIters][kTouchLines];
    select_and_build(keys, n, N, nullptr, 0, nullptr, 0, keep, H, (p.off_lists - p.off_keys) / 4, nullptr, nullptr,
                     0u, 0, tch);
}

// Standalone gather from a keep mask.
template <int DT, int D>
__global__ void __launch_bounds__(NT) compact_kernel(const UnitParams p) {
    using S = Shape<DT, D>;
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    uint32_t *holes = reinterpret_cast<uint32_t *>(lds + p.off_lists);
    uint32_t *movers = holes + p.evict_cap;
    const int head = blockIdx.x, layer = blockIdx.y, sl = blockIdx.z;
    const int ul = (sl * p.num_layers + layer) * p.num_kv_heads + head;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl], N = p.nN[2 * sl + 1];
    if (n <= N) return;
    const int64_t cap = p.capacity;
    const uint8_t *keep = p.keep_in + u * cap;
    // wave-segmented ranks of holes (slots < N, not kept) and movers (slots >= N, kept)
    const int w = wave_id(), lane = lane_id();
    const int seg = (((n + NW - 1) / NW) + 63) & ~63;
    const int j0 = w * seg, j1 = min(n, j0 + seg);
    uint32_t ch = 0, cm = 0;
    for (int jb = j0; jb < j1; jb += 64) {
        const int j = jb + lane;
        const bool kp = j < j1 && keep[j] != 0;
        ch += __popcll(__ballot(j < j1 && j < N && !kp));
        cm += __popcll(__ballot(kp && j >= N));
    }
    if (lane == 0) {
        H.bc[w] = ch;
        H.bc[32 + w] = cm;
    }
    __syncthreads();
    uint32_t h_off = 0, m_off = 0, h_tot = 0, m_tot = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        h_off += i < w ? H.bc[i] : 0u;
        m_off += i < w ? H.bc[32 + i] : 0u;
        h_tot += H.bc[i];
        m_tot += H.bc[32 + i];
    }
    for (int jb = j0; jb < j1; jb += 64) {
        const int j = jb + lane;
        const bool kp = j < j1 && keep[j] != 0;
        const bool hole = j < j1 && j < N && !kp;
        const bool mover = kp && j >= N;
        const uint64_t mh = __ballot(hole), mm = __ballot(mover);
        const uint32_t rh = h_off + __popcll(mh & lanes_below());
        const uint32_t rm = m_off + __popcll(mm & lanes_below());
        if (hole && rh < (uint32_t)p.evict_cap) holes[lds_ix<kSiteLists>((int)rh, p.evict_cap)] = (uint32_t)j;
        if (mover && rm < (uint32_t)p.move_cap) movers[lds_ix<kSiteLists>((int)rm, p.move_cap)] = (uint32_t)j;
        h_off += __popcll(mh);
        m_off += __popcll(mm);
    }
    __syncthreads();
    int moves = (int)min(h_tot, m_tot);
    moves = min(moves, min(p.evict_cap, p.move_cap));
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    char *kb = p.k ? p.k + off : nullptr;
    char *vb = p.v + off;
    int32_t *pos = p.pos ? p.pos + u * cap : nullptr;
    const uint32_t ss32 = p.s_slot;
    const int cl = lane % S::LPR;
    const int g = wave_id() * S::RPW + lane / S::LPR;
    for (int e = g; e < moves; e += S::GROUPS) {
        const int dst = (int)holes[lds_ix<kSiteLists>(e, p.evict_cap)];
        const int src = (int)movers[lds_ix<kSiteLists>(e, p.move_cap)];
        const uint4 kv = kb ? load_stream(kb, row_off(src, ss32, cl)) : make_uint4(0u, 0u, 0u, 0u);
        const uint4 vv = load_stream(vb, row_off(src, ss32, cl));
        if (kb) store_stream(kb, row_off(dst, ss32, cl), kv);
        store_stream(vb, row_off(dst, ss32, cl), vv);
        if (pos && cl == 0) pos[dst] = pos[src];
    }
}

// ---------------------------------------------------------------- geometry

// Wave-wide fp64 sum by butterfly: every lane ends with the same bits.
__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// Element c of a row as fp32.
template <int DT> __device__ __forceinline__ float row_elem(const char *row, int c) {
    if constexpr (DT == 0)
        return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(row)[c] << 16);
    else
        return reinterpret_cast<const float *>(row)[c];
}

// Geometry of one unit's keys and values (Sec. 3.1, and the bos-cosim of
// Sec. 4): for K and for V, the mean distance of the n rows to their centroid
// and the population standard deviation of those distances; and the cosine
// between the first key and the mean of the other keys.  Every distance needs
// the centroid of all n rows.  When the caller supplies the column sums of K
// and V over exactly the n rows (k_sum, v_sum with count n: the pass keeps
// V's as its running sum), the centroids are known up front and one stream
// over the rows gives every distance; otherwise a first stream sums the
// columns in fp64 and a second one takes the distances.  A distance is taken
// in fp32 from the difference to the centroid held as an fp32 pair (hi +
// lo), so that its error stays at fp32 rounding of the distance however far
// the centroid lies from the origin; every sum over rows is fp64, in a fixed
// order.  With two streams the first keeps the rows cacheable and the second
// reads them once more, in reverse order and without retention.
constexpr int kGeoRows = 2;  // rows per lane group in one tile of the geometry streams

template <int DT, int D>
__global__ void __launch_bounds__(NT) geometry_kernel(const UnitParams p) {
    using S = Shape<DT, D>;
    using E = Elem<DT>;
    constexpr int kTile = S::GROUPS * kGeoRows;  // rows per tile
    extern __shared__ __align__(16) unsigned char lds[];
    LdsHead &H = *reinterpret_cast<LdsHead *>(lds);
    double *red = reinterpret_cast<double *>(lds + p.off_keys);  // NW*D doubles
    float *ctr = reinterpret_cast<float *>(lds + p.off_lists);   // K hi, K lo, V hi, V lo: D each

    const int head = blockIdx.x, layer = blockIdx.y, sl = blockIdx.z;
    const int ul = (sl * p.num_layers + layer) * p.num_kv_heads + head;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl];
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    const char *kb = p.k + off;
    const char *vb = p.v + off;
    const uint32_t ss32 = p.s_slot;
    double *out = p.geom_out + u * 5;
    const int lane = lane_id(), w = wave_id();
    const int cl = lane % S::LPR;
    const int g = w * S::RPW + lane / S::LPR;  // this lane's row group
    if (n == 0) {
        if (threadIdx.x < 5) out[threadIdx.x] = 0.0;
        return;
    }

    // Both streams keep one tile of 2 * kGeoRows 16-byte chunks in flight per
    // lane (chunk j: row j/2 of the tile's kGeoRows rows of this lane's group;
    // K for even j, V for odd j).  A chunk is refilled with the next tile's as soon
    // as it is used; the refill's address depends on the used values, so the
    // loads stay in order and each use waits for its own chunk only.  The
    // tile after the last is requested too, with rows clamped into [0, n).
    uint4 buf[2 * kGeoRows];
    auto chunk_off = [&](int e0, int j, uint32_t z) __attribute__((always_inline)) {
        return row_off(min(max(e0, 0) + (j >> 1) * S::GROUPS + g, n - 1), ss32, cl) + z;
    };

    // ---- centroids: the caller's column sums when they cover the n rows,
    // else fp64 column sums of all n rows (a first stream) ----
    const double *ksu = p.k_sum ? p.k_sum + u * (D + 1) : nullptr;
    const double *vsu = p.v_sum ? p.v_sum + u * (D + 1) : nullptr;
    // the distance stream's first tile (its last rows) goes out at once when
    // sums are given, before their counts arrive: it does not depend on them
    const int last = ((n - 1) / kTile) * kTile;
    auto first_distance_tile = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < 2 * kGeoRows; ++j) {
            buf[j] = load_stream((j & 1) ? vb : kb, chunk_off(last, j, 0u));
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    if (ksu && vsu) first_distance_tile();
    const bool given = ksu && vsu && ksu[D] == (double)n && vsu[D] == (double)n;  // uniform
    double sk = 0.0, sv = 0.0;
    if (given) {
        if (threadIdx.x < D) {
            sk = ksu[threadIdx.x];
            sv = vsu[threadIdx.x];
        }
    } else {
        double ak[S::EPL], av[S::EPL];
#pragma unroll
        for (int i = 0; i < S::EPL; ++i) ak[i] = av[i] = 0.0;
#pragma unroll
        for (int j = 0; j < 2 * kGeoRows; ++j) {
            buf[j] = *reinterpret_cast<const uint4 *>(((j & 1) ? vb : kb) + chunk_off(0, j, 0u));
            __builtin_amdgcn_sched_barrier(0);  // issued in chunk order, as the loop reissues them
        }
        for (int e0 = 0; e0 < n; e0 += kTile) {
#pragma unroll
            for (int r = 0; r < kGeoRows; ++r) {
                float x[S::EPL], y[S::EPL];
                E::unpack(buf[2 * r], x);
                E::unpack(buf[2 * r + 1], y);
                const bool valid = e0 + r * S::GROUPS + g < n;  // selects, not a branch
#pragma unroll
                for (int i = 0; i < S::EPL; ++i) {
                    ak[i] += valid ? (double)x[i] : 0.0;
                    av[i] += valid ? (double)y[i] : 0.0;
                }
                const uint32_t z = zero_after(x[0] + y[0]);
                buf[2 * r] = *reinterpret_cast<const uint4 *>(kb + chunk_off(e0 + kTile, 2 * r, z));
                buf[2 * r + 1] = *reinterpret_cast<const uint4 *>(vb + chunk_off(e0 + kTile, 2 * r + 1, z));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        const int red_cap = (p.off_lists - p.off_keys) / 8;
        sk = block_col_total<DT, D>(ak, red, red_cap);
        __syncthreads();  // every column total of K is read before red is refilled
        sv = block_col_total<DT, D>(av, red, red_cap);
    }

    // centroid pairs for the distance stream, and the bos-cosim terms:
    // k_0 . m, |k_0|^2, |m|^2 with m the mean of keys 1 .. n-1
    double bos_dot = 0.0, bos_k0 = 0.0, bos_m = 0.0;
    if (threadIdx.x < D) {
        const int t = threadIdx.x;
        const double mk = sk / (double)n, mv = sv / (double)n;
        const float kh = (float)mk, vh = (float)mv;
        ctr[t] = kh;
        ctr[D + t] = (float)(mk - (double)kh);
        ctr[2 * D + t] = vh;
        ctr[3 * D + t] = (float)(mv - (double)vh);
        if (n >= 2) {
            const double k0 = (double)row_elem<DT>(kb, t);
            const double m = (sk - k0) / (double)(n - 1);
            bos_dot = k0 * m;
            bos_k0 = k0 * k0;
            bos_m = m * m;
        }
    }
    bos_dot = wave_sum_f64(bos_dot);
    bos_k0 = wave_sum_f64(bos_k0);
    bos_m = wave_sum_f64(bos_m);
    if (lane == 0) {
        H.old_sum[3 * w] = bos_dot;
        H.old_sum[3 * w + 1] = bos_k0;
        H.old_sum[3 * w + 2] = bos_m;
    }
    __syncthreads();

    // ---- distances ----
    float kh[S::EPL], kl[S::EPL], vh[S::EPL], vl[S::EPL];
#pragma unroll
    for (int i = 0; i < S::EPL; ++i) {
        const int c = cl * S::EPL + i;
        kh[i] = ctr[c];
        kl[i] = ctr[D + c];
        vh[i] = ctr[2 * D + c];
        vl[i] = ctr[3 * D + c];
    }
    double s1k = 0.0, s2k = 0.0, s1v = 0.0, s2v = 0.0;
    // last tile first: the rows a first stream read most recently are the
    // likeliest still to be held in the caches
    if (!given) first_distance_tile();
    for (int e0 = last; e0 >= 0; e0 -= kTile) {
#pragma unroll
        for (int r = 0; r < kGeoRows; ++r) {
            float x[S::EPL], y[S::EPL];
            E::unpack(buf[2 * r], x);
            E::unpack(buf[2 * r + 1], y);
            float a = 0.f, b = 0.f;
#pragma unroll
            for (int i = 0; i < S::EPL; ++i) {
                const float dx = (x[i] - kh[i]) - kl[i];
                const float dy = (y[i] - vh[i]) - vl[i];
                a = fmaf(dx, dx, a);
                b = fmaf(dy, dy, b);
            }
            const uint32_t z = zero_after(a + b);
            buf[2 * r] = load_stream(kb, chunk_off(e0 - kTile, 2 * r, z));
            buf[2 * r + 1] = load_stream(vb, chunk_off(e0 - kTile, 2 * r + 1, z));
            __builtin_amdgcn_sched_barrier(0);
            const double dk = (double)score_sqrt(row_sum<S::LPR>(a));
            const double dv = (double)score_sqrt(row_sum<S::LPR>(b));
            const bool mine = cl == 0 && e0 + r * S::GROUPS + g < n;  // one lane per row
            s1k += mine ? dk : 0.0;
            s2k += mine ? dk * dk : 0.0;
            s1v += mine ? dv : 0.0;
            s2v += mine ? dv * dv : 0.0;
        }
    }
    s1k = wave_sum_f64(s1k);
    s2k = wave_sum_f64(s2k);
    s1v = wave_sum_f64(s1v);
    s2v = wave_sum_f64(s2v);
    if (lane == 0) {  // red was last read before the barrier above
        red[4 * w] = s1k;
        red[4 * w + 1] = s2k;
        red[4 * w + 2] = s1v;
        red[4 * w + 3] = s2v;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double t[4] = {0.0, 0.0, 0.0, 0.0}, b[3] = {0.0, 0.0, 0.0};
        for (int ww = 0; ww < NW; ++ww) {
#pragma unroll
            for (int j = 0; j < 4; ++j) t[j] += red[4 * ww + j];
#pragma unroll
            for (int j = 0; j < 3; ++j) b[j] += H.old_sum[3 * ww + j];
        }
        const double inv_n = 1.0 / (double)n;
        const double muk = t[0] * inv_n, muv = t[2] * inv_n;
        // population variance of the distances, E[d^2] - E[d]^2 in fp64
        out[0] = sqrt(fmax(t[1] * inv_n - muk * muk, 0.0));
        out[1] = sqrt(fmax(t[3] * inv_n - muv * muv, 0.0));
        out[2] = muk;
        out[3] = muv;
        const double den = sqrt(b[1]) * sqrt(b[2]);
        out[4] = den > 0.0 ? b[0] / den : 0.0;
    }
}

template <int DT> void *geometry_kernel_for(int head_dim) {
    switch (head_dim) {
        case 64: return reinterpret_cast<void *>(&geometry_kernel<DT, 64>);
        case 128: return reinterpret_cast<void *>(&geometry_kernel<DT, 128>);
        case 256: return reinterpret_cast<void *>(&geometry_kernel<DT, 256>);
    }
    return nullptr;
}

// ---------------------------------------------------------------- decode attention

// One decode step of the newest token of every sequence fused with its
// eviction (Sec. 2.1, Eq. attention and Eq. eviction, with B = 1 in Eq.
// block_processing): the query rows of the G query heads that share a KV head
// attend to all n cached rows, and the same stream over V scores every row
// against the mean that the running sum gives (Sec. 3.2, Eq. vd), so that the
// eviction needs no V read of its own.  A unit's rows are split over several
// workgroups (split kernel); a second kernel merges the splits, evicts the row
// with the lowest score when n = N + 1, moves the newest row into its slot and
// updates the running sum.  (A merge by the last split to finish needs a
// device-scope release per workgroup, which writes back the XCD's L2 and was
// measured several times slower.)
//
// Softmax runs in log2 units (the query is pre-scaled by scale * log2(e)) with
// a running reference: every lane group keeps, per head, a reference logit,
// the sum of 2^(z - reference) and the weighted sum of its value columns,
// rescaled when the reference is raised; two rows are taken at a time.
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr float kNoLogit = -1.0e30f;  // below every logit, finite (2^(kNoLogit - z) = 0)
constexpr int kAttnRows = 2;           // rows per lane group in one tile of the split kernel
// Lazy rescaling: a lane group's softmax reference (its largest logit so far,
// in log2 units) is raised only when a logit exceeds it by more than this, so
// every weight 2^(z - reference) stays at most 2^8 and most tiles leave the
// running sums unscaled.  The merges take each part's reference, whatever it is.
constexpr float kLazyLog2 = 8.0f;
constexpr int kMergeBatch = 8;  // splits whose partials the combine loads at once

template <int DT, int D> struct AttnShape {
    static constexpr int EPL = Elem<DT>::EPL;
    static constexpr int ROWB = D * Elem<DT>::BYTES;
    static constexpr int LPR = ROWB / 16;
    static constexpr int RPW = 64 / LPR;
    static constexpr int GROUPS = kAttnWaves * RPW;   // row groups of a workgroup
    static constexpr int TILE = kAttnRows * GROUPS;   // rows per tile
};

// fp64 mean of a unit's n rows from the running sum (count rows) plus the rows
// [count, n) read here, as a pair of fp32 numbers: its rounding into
// mean[0 .. D) and the rest into mean_lo[0 .. D); thread t < D takes column t.
template <int DT, int D>
__device__ __forceinline__ void attn_mean(const double *st, const char *vb, uint32_t ss, int n,
                                          int count, float *mean, float *mean_lo) {
    if (threadIdx.x < D) {
        const int t = threadIdx.x;
        double f = 0.0;
        for (int r = count; r < n; ++r) f += (double)row_elem<DT>(vb + (size_t)r * ss, t);
        const double old = count > 0 ? st[t] : 0.0;
        const double m = (old + f) / (double)n;
        const float hi = (float)m;
        mean[t] = hi;
        mean_lo[t] = (float)(m - (double)hi);
    }
}

__device__ __forceinline__ int state_count(const double *st, int n) {
    const double c = st[0];
    return (c >= 0.0 && c <= (double)n && c == (double)(int)c) ? (int)c : 0;
}

// CAOTE: the FastCAOTE variant (App. A, Eq. app_fastcaote), whose score needs
// every row's weight under the merged softmax: each row's G logits (log2
// units) and its distance to the mean are kept in LDS, rows[(e - r0) * (G+1)
// + g] and [.. + G], and written to the workspace at the split's end, for the
// combine kernel to score once the splits' maxima and sums are merged.
template <int DT, int D, int G, bool CAOTE>
__global__ void __launch_bounds__(kAttnThreads) attn_split_kernel(const UnitParams p) {
    using A = AttnShape<DT, D>;
    using E = Elem<DT>;
    constexpr int EPL = A::EPL, LPR = A::LPR, GROUPS = A::GROUPS;
    extern __shared__ __align__(16) unsigned char lds[];
    float *mean = reinterpret_cast<float *>(lds);                          // D
    float *mean_lo = mean + D;                                             // D
    float *gmax = mean_lo + D;                                             // GROUPS * G
    float *gsum = gmax + GROUPS * G;                                       // GROUPS * G
    unsigned long long *wmin = reinterpret_cast<unsigned long long *>(gsum + GROUPS * G);  // kAttnWaves
    float *red = reinterpret_cast<float *>(wmin + kAttnWaves);             // G * GROUPS * D
    float *rows = red + G * GROUPS * D;                                    // CAOTE: split_rows * (G + 1)

    const int sp = blockIdx.x, head = blockIdx.y;
    const int sl = blockIdx.z / p.num_layers, layer = blockIdx.z % p.num_layers;
    const int ul = (sl * p.num_layers + layer) * p.num_kv_heads + head;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl];
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    const char *kb = p.k + off;
    const char *vb = p.v + off;
    const uint32_t ss32 = p.s_slot;
    const double *st = p.running_sum + u * (D + 1);
    const int lane = lane_id(), w = wave_id();
    const int cl = lane % LPR;
    const int grp = w * A::RPW + lane / LPR;
    const int r0 = sp * p.split_rows;
    const int r1 = min(n, r0 + p.split_rows);
    const int64_t wsi = u * p.splits + sp;

    if (r1 > r0) attn_mean<DT, D>(st, vb, ss32, n, state_count(st + D, n), mean, mean_lo);
    // this lane's columns of the G query rows, pre-scaled
    float qs[G][EPL];
    const float *qrow = p.q + (((int64_t)sl * p.num_layers + layer) * p.num_kv_heads + head) * G * D;
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < EPL; ++i) qs[g][i] = qrow[g * D + cl * EPL + i] * p.qscale;
    __syncthreads();
    float mv[EPL], mvl[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
        mv[i] = mean[cl * EPL + i];
        mvl[i] = mean_lo[cl * EPL + i];
    }

    float mx[G], ls[G], acc[G][EPL];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        mx[g] = kNoLogit;
        ls[g] = 0.f;
#pragma unroll
        for (int i = 0; i < EPL; ++i) acc[g][i] = 0.f;
    }
    unsigned long long amin = ~0ull;

    // Rows of 16 lanes (bf16 with d = 128, fp32 with d = 64): the tile's
    // 2 * (G + 1) row sums (G logits and a distance per row) are reduced
    // together, each exchange leaving every lane with half as many values:
    // the row's lower half keeps row 0 and its upper half row 1 (row_mirror),
    // then the even and odd banks of four lanes keep the two heads of a pair
    // (row_half_mirror), then the quad sums.  Bank k = (lane % 16) / 4 then
    // holds row k / 2: head k % 2 (and, with G = 4, head 2 + k % 2) and the
    // distance.  Each bank takes its weights' exponentials once, and every
    // lane receives all of them by row_newbcast from the first lane of each
    // bank.
    constexpr bool kPacked = LPR == 16 && kAttnRows == 2;
    constexpr int NQ = G == 4 ? 2 : 1;  // logits per lane after the reduction
    // With G = 4 the weighted sum of the value rows runs on the matrix cores:
    // v_mfma_f32_4x4x1_16b_f32 treats each quad of lanes as a block whose
    // 4 x 4 outer product adds (the weight of head i from lane i of the quad)
    // x (the value of lane j) to row i of lane j.  With lane i of each quad
    // holding head i's weight and every lane its own value column, accv[k][g]
    // is acc[g][k]: the same sums, each rounded once per row as the fused
    // multiply-add chain it replaces.
    constexpr bool kMfma = kPacked && G == 4;
    f32x4 accv[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) accv[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int bank = (lane & 15) >> 2;
    const bool upper = bank >= 2, odd = (bank & 1) != 0;
    const int rb = upper ? 1 : 0;  // this lane's row of the tile after the reduction
    int hq[NQ];                    // and its heads
#pragma unroll
    for (int h = 0; h < NQ; ++h) hq[h] = G == 1 ? 0 : 2 * h + (odd ? 1 : 0);
    // the references of this lane's heads, and its part of their weight sums
    // (the weights of row rb only; the row's other half holds the rest)
    float mxq[NQ], lsq[NQ];
#pragma unroll
    for (int h = 0; h < NQ; ++h) {
        mxq[h] = kNoLogit;
        lsq[h] = 0.f;
    }
    // nx[r]: this lane's byte offset in row r of the next tile to load (the
    // last row of the split stands in past its end)
    const uint32_t tile_bytes = (uint32_t)A::TILE * ss32, lim_off = row_off(max(r1 - 1, 0), ss32, cl);
    uint32_t nx[kAttnRows];
#pragma unroll
    for (int r = 0; r < kAttnRows; ++r) nx[r] = row_off(r0 + r * GROUPS + grp, ss32, cl) + tile_bytes;
    auto packed_tile = [&](int e0, uint4 (&buf)[2 * kAttnRows]) __attribute__((always_inline)) {
        float a[kAttnRows][G], b[kAttnRows], vx[kAttnRows][EPL];
#pragma unroll
        for (int r = 0; r < kAttnRows; ++r) {
            float kx[EPL];
            E::unpack(buf[2 * r], kx);
            E::unpack(buf[2 * r + 1], vx[r]);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                a[r][g] = 0.f;
#pragma unroll
                for (int i = 0; i < EPL; ++i) a[r][g] = fmaf(qs[g][i], kx[i], a[r][g]);
            }
            b[r] = 0.f;
#pragma unroll
            for (int i = 0; i < EPL; ++i) {
                const float t = (vx[r][i] - mv[i]) - mvl[i];
                b[r] = fmaf(t, t, b[r]);
            }
            // refill both chunks of this row with the next tile's
            const uint32_t o = min(nx[r], lim_off) + zero_after(a[r][0] + b[r]);
            nx[r] += tile_bytes;
            buf[2 * r] = load_stream(kb, o);
            buf[2 * r + 1] = load_stream(vb, o);
            __builtin_amdgcn_sched_barrier(0);
        }
        // row_mirror: the lower half keeps row 0, the upper half row 1
        float pr[G], pd;
#pragma unroll
        for (int g = 0; g < G; ++g)
            pr[g] = (upper ? a[1][g] : a[0][g]) + dpp<0x140>(upper ? a[0][g] : a[1][g]);
        pd = (upper ? b[1] : b[0]) + dpp<0x140>(upper ? b[0] : b[1]);
        // row_half_mirror: even banks keep the pair's first head, odd banks the second
        float q[NQ];
        if constexpr (G == 1) {
            q[0] = pr[0] + dpp<0x141>(pr[0]);
        } else {
#pragma unroll
            for (int h = 0; h < NQ; ++h)
                q[h] = (odd ? pr[2 * h + 1] : pr[2 * h]) + dpp<0x141>(odd ? pr[2 * h] : pr[2 * h + 1]);
        }
        pd += dpp<0x141>(pd);
#pragma unroll
        for (int h = 0; h < NQ; ++h) {
            q[h] += dpp<0x4E>(q[h]);  // quad_perm [2,3,0,1]
            q[h] += dpp<0xB1>(q[h]);  // quad_perm [1,0,3,2]
        }
        pd += dpp<0x4E>(pd);
        pd += dpp<0xB1>(pd);
        // this lane's logits: head hq[h] of row rb
        const int e = e0 + rb * GROUPS + grp;
        const bool vr = e < r1;
        float zq[NQ];
#pragma unroll
        for (int h = 0; h < NQ; ++h) zq[h] = vr ? q[h] : kNoLogit;
        // L2 score of the value row (Sec. 3.2, Eq. vd) and its key
        const float dist = score_sqrt(pd);
        if constexpr (CAOTE) {  // the row's logits and distance, for the combine
            if ((lane & 3) == 0 && vr) {
#pragma unroll
                for (int h = 0; h < NQ; ++h)
                    if (G != 1 || !odd)
                        rows[lds_ix<kSiteRows>((e - r0) * (G + 1) + hq[h], p.split_rows * (G + 1))] = zq[h];
                if (!odd) rows[lds_ix<kSiteRows>((e - r0) * (G + 1) + G, p.split_rows * (G + 1))] = dist;
            }
        } else {
            const uint32_t key = score_key(dist);
            const unsigned long long pk = ((unsigned long long)key << 32) | (uint32_t)~(uint32_t)e;
            amin = vr && pk < amin ? pk : amin;
        }
        // the lazy raise of the references (a wave-uniform branch)
        bool grow = false;
#pragma unroll
        for (int h = 0; h < NQ; ++h) grow = grow || zq[h] > mxq[h] + kLazyLog2;
        if (__builtin_amdgcn_ballot_w64(grow)) {
            // every logit of the tile to every lane of its row group
            float zall[kAttnRows][G];
            static_for<4>([&](auto kc) __attribute__((always_inline)) {
                constexpr int k = decltype(kc)::value;
#pragma unroll
                for (int h = 0; h < NQ; ++h) {
                    const float zb = row_bcast<4 * k>(zq[h]);
                    if (G != 1 || (k & 1) == 0) zall[k >> 1][G == 1 ? 0 : 2 * h + (k & 1)] = zb;
                }
            });
            float cg[G];
#pragma unroll
            for (int g = 0; g < G; ++g) {
                float mn = mx[g];
#pragma unroll
                for (int r = 0; r < kAttnRows; ++r) mn = fmaxf(mn, zall[r][g]);
                cg[g] = __builtin_amdgcn_exp2f(mx[g] - mn);
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    if constexpr (kMfma)
                        accv[i][g] *= cg[g];
                    else
                        acc[g][i] *= cg[g];
                }
                mx[g] = mn;
            }
#pragma unroll
            for (int h = 0; h < NQ; ++h) {
                float c = cg[0], m = mx[0];
#pragma unroll
                for (int g = 1; g < G; ++g) {
                    c = hq[h] == g ? cg[g] : c;
                    m = hq[h] == g ? mx[g] : m;
                }
                lsq[h] *= c;
                mxq[h] = m;
            }
        }
        // the weights: one exponential per bank and head (an invalid row's
        // exponent underflows to 0), then to every lane
        float wq[NQ];
#pragma unroll
        for (int h = 0; h < NQ; ++h) {
            wq[h] = __builtin_amdgcn_exp2f(vr ? zq[h] - mxq[h] : kNoLogit);
            lsq[h] += wq[h];
        }
        float w[kAttnRows][G];
        static_for<4>([&](auto kc) __attribute__((always_inline)) {
            constexpr int k = decltype(kc)::value;
            if constexpr (G == 4) {  // the bank's two weights as one 64-bit move
                const long pair = ((long)__float_as_int(wq[NQ - 1]) << 32) | (uint32_t)__float_as_int(wq[0]);
                const long got = row_bcast<4 * k>(pair);
                w[k >> 1][k & 1] = __int_as_float((int)(uint32_t)got);
                w[k >> 1][(2 + (k & 1)) % G] = __int_as_float((int)(got >> 32));
            } else if constexpr (G == 2 || (k & 1) == 0) {
                w[k >> 1][G == 1 ? 0 : (k & 1) % G] = row_bcast<4 * k>(wq[0]);
            }
        });
        if constexpr (kMfma) {
            // lane i of each quad feeds in head i's weight: head i of row r is
            // in bank 2r + (i & 1), in the high word of its pair when i >= 2
            const long pair = ((long)__float_as_int(wq[1]) << 32) | (uint32_t)__float_as_int(wq[0]);
            const bool odd_head = (lane & 1) != 0, high_head = (lane & 2) != 0;
            long b0 = row_bcast<0>(pair), b1 = row_bcast<4>(pair), b2 = row_bcast<8>(pair), b3 = row_bcast<12>(pair);
            // every lane takes part in all four broadcasts (a select between
            // two broadcasts may otherwise become a branch, each broadcast
            // then reading lanes the branch has switched off)
            asm volatile("" : "+v"(b0), "+v"(b1), "+v"(b2), "+v"(b3));
            const long p0 = odd_head ? b1 : b0;
            const long p1 = odd_head ? b3 : b2;
            const float wa[kAttnRows] = {__int_as_float((int)(high_head ? (uint32_t)(p0 >> 32) : (uint32_t)p0)),
                                         __int_as_float((int)(high_head ? (uint32_t)(p1 >> 32) : (uint32_t)p1))};
#pragma unroll
            for (int r = 0; r < kAttnRows; ++r)
#pragma unroll
                for (int i = 0; i < EPL; ++i)
                    accv[i] = __builtin_amdgcn_mfma_f32_4x4x1f32(wa[r], vx[r][i], accv[i], 0, 0, 0);
        } else {
#pragma unroll
            for (int g = 0; g < G; ++g) {
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    float x = acc[g][i];
#pragma unroll
                    for (int r = 0; r < kAttnRows; ++r) x = fmaf(w[r][g], vx[r][i], x);
                    acc[g][i] = x;
                }
            }
        }
    };

    if (r1 > r0) {
        // chunk j of a tile: row j/2 of this group's kAttnRows rows, K for even j, V for odd
        uint4 buf[2 * kAttnRows];
        auto chunk_off = [&](int e0, int j, uint32_t z) __attribute__((always_inline)) {
            return row_off(min(e0 + (j >> 1) * GROUPS + grp, r1 - 1), ss32, cl) + z;
        };
#pragma unroll
        for (int j = 0; j < 2 * kAttnRows; ++j) {
            buf[j] = load_stream((j & 1) ? vb : kb, chunk_off(r0, j, 0u));
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (kPacked) {
            for (int e0 = r0; e0 < r1; e0 += A::TILE) packed_tile(e0, buf);
        }
        if constexpr (!kPacked) {
          for (int e0 = r0; e0 < r1; e0 += A::TILE) {
            float z[kAttnRows][G], vx[kAttnRows][EPL];
            bool valid[kAttnRows];
#pragma unroll
            for (int r = 0; r < kAttnRows; ++r) {
                float kx[EPL];
                E::unpack(buf[2 * r], kx);
                E::unpack(buf[2 * r + 1], vx[r]);
                const int e = e0 + r * GROUPS + grp;
                valid[r] = e < r1;
                float a[G];
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    a[g] = 0.f;
#pragma unroll
                    for (int i = 0; i < EPL; ++i) a[g] = fmaf(qs[g][i], kx[i], a[g]);
                }
                float b = 0.f;
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    const float t = (vx[r][i] - mv[i]) - mvl[i];
                    b = fmaf(t, t, b);
                }
                // refill both chunks of this row with the next tile's
                const uint32_t zz = zero_after(a[0] + b);
                buf[2 * r] = load_stream(kb, chunk_off(e0 + A::TILE, 2 * r, zz));
                buf[2 * r + 1] = load_stream(vb, chunk_off(e0 + A::TILE, 2 * r + 1, zz));
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int g = 0; g < G; ++g) z[r][g] = valid[r] ? row_sum<LPR>(a[g]) : kNoLogit;
                // L2 score of the value row (Sec. 3.2, Eq. vd) and its key
                const float dist = score_sqrt(row_sum<LPR>(b));
                if constexpr (CAOTE) {  // the row's logits and distance, for the combine
                    if (cl == 0 && valid[r]) {
#pragma unroll
                        for (int g = 0; g < G; ++g)
                            rows[lds_ix<kSiteRows>((e - r0) * (G + 1) + g, p.split_rows * (G + 1))] = z[r][g];
                        rows[lds_ix<kSiteRows>((e - r0) * (G + 1) + G, p.split_rows * (G + 1))] = dist;
                    }
                } else {
                    const uint32_t key = score_key(dist);
                    const unsigned long long pk = ((unsigned long long)key << 32) | (uint32_t)~(uint32_t)e;
                    amin = valid[r] && pk < amin ? pk : amin;
                }
            }
            // the reference moves only when a logit passes it by more than
            // kLazyLog2 (a wave-uniform branch, taken by few tiles)
            bool grow = false;
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int r = 0; r < kAttnRows; ++r) grow = grow || z[r][g] > mx[g] + kLazyLog2;
            if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    float mn = mx[g];
#pragma unroll
                    for (int r = 0; r < kAttnRows; ++r) mn = fmaxf(mn, z[r][g]);
                    const float c = __builtin_amdgcn_exp2f(mx[g] - mn);
#pragma unroll
                    for (int i = 0; i < EPL; ++i) acc[g][i] *= c;
                    ls[g] *= c;
                    mx[g] = mn;
                }
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                float w[kAttnRows], ws = 0.f;
#pragma unroll
                for (int r = 0; r < kAttnRows; ++r) {
                    w[r] = valid[r] ? __builtin_amdgcn_exp2f(z[r][g] - mx[g]) : 0.f;
                    ws += w[r];
                }
#pragma unroll
                for (int i = 0; i < EPL; ++i) {
                    float x = acc[g][i];
#pragma unroll
                    for (int r = 0; r < kAttnRows; ++r) x = fmaf(w[r], vx[r][i], x);
                    acc[g][i] = x;
                }
                ls[g] += ws;
            }
          }
        }
    }
    if constexpr (kMfma)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int i = 0; i < EPL; ++i) acc[g][i] = accv[i][g];
    if constexpr (kPacked) {  // head g's weight sum: rows 0 and 1, from banks g % 2 and g % 2 + 2
        static_for<G>([&](auto gc) __attribute__((always_inline)) {
            constexpr int g = decltype(gc)::value;
            constexpr int k0 = G == 1 ? 0 : g % 2;
            ls[g] = row_bcast<4 * k0>(lsq[g / 2]) + row_bcast<4 * k0 + 8>(lsq[g / 2]);
        });
    }

    // merge the row groups: per head the largest logit, then the rescaled sums
    // in a fixed order
    if (cl == 0)
#pragma unroll
        for (int g = 0; g < G; ++g) gmax[grp * G + g] = mx[g];
    amin = wave_min_u64(amin);
    if (lane == 0) wmin[w] = amin;
    __syncthreads();
#pragma unroll
    for (int g = 0; g < G; ++g) {
        float top = kNoLogit;
        for (int q = 0; q < GROUPS; ++q) top = fmaxf(top, gmax[q * G + g]);
        const float f = __builtin_amdgcn_exp2f(mx[g] - top);
#pragma unroll
        for (int i = 0; i < EPL; ++i) red[(g * GROUPS + grp) * D + cl * EPL + i] = acc[g][i] * f;
        if (cl == 0) gsum[grp * G + g] = ls[g] * f;
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * D; idx += kAttnThreads) {
        const int g = idx / D, c = idx % D;
        float s = 0.f;
        for (int q = 0; q < GROUPS; ++q) s += red[(g * GROUPS + q) * D + c];
        p.ws_acc[(wsi * G + g) * D + c] = s;
    }
    if (threadIdx.x < G) {
        const int g = threadIdx.x;
        float top = kNoLogit, l = 0.f;
        for (int q = 0; q < GROUPS; ++q) top = fmaxf(top, gmax[q * G + g]);
        for (int q = 0; q < GROUPS; ++q) l += gsum[q * G + g];
        p.ws_ml[(wsi * G + g) * 2] = top;
        p.ws_ml[(wsi * G + g) * 2 + 1] = l;
    }
    if (threadIdx.x == 0) {
        unsigned long long m = ~0ull;
        for (int q = 0; q < kAttnWaves; ++q) m = wmin[q] < m ? wmin[q] : m;
        p.ws_amin[wsi] = m;
    }
    if constexpr (CAOTE) {  // the rows' logits and distances (written before the barrier above)
        const int cnt = max(r1 - r0, 0) * (G + 1);
        float *dst = p.ws_rows + (u * p.capacity + r0) * (G + 1);
        for (int i = threadIdx.x; i < cnt; i += kAttnThreads)
            dst[i] = rows[lds_ix<kSiteRows>(i, p.split_rows * (G + 1))];
    }
}

// FastCAOTE scores of a unit's rows (App. A, Eq. app_fastcaote) from the
// logits and distances its splits stored, and their minimum as (key << 32 |
// ~slot), the lowest score and the highest slot among equal ones: a_j = (1/G)
// sum_g 2^(z_gj - M_g) / L_g with M_g, L_g the merged maximum and weight sum
// of head g, 1 - a_j = (1/G) sum_g (L_g - w_gj) / L_g (a row that holds all
// of a head's weight scores +infinity).  Every thread of the block takes part
// and receives the minimum; `ml` is the unit's [S][G][2] split maxima and sums.
template <int G>
__device__ __forceinline__ unsigned long long caote_argmin(const UnitParams &p, int64_t u, int n,
                                                           const float *ml, int S) {
    __shared__ float mg[G], lg[G];
    __shared__ unsigned long long wbest[kAttnWaves];
    // kRowsAtOnce rows per thread at a time, all their words read before any
    // is used (one memory round trip per batch; n = 4097 is one batch), the
    // first batch before the heads' maxima and sums are merged
    constexpr int kRowsAtOnce = 17;
    const float *rows = p.ws_rows + u * p.capacity * (G + 1);
    float x[kRowsAtOnce][G + 1];
    auto load_rows = [&](int j0) __attribute__((always_inline)) {
#pragma unroll
        for (int r = 0; r < kRowsAtOnce; ++r) {
            const int j = min(j0 + r * kAttnThreads, n - 1);  // past the end: row n - 1 again, unused
#pragma unroll
            for (int g = 0; g <= G; ++g) x[r][g] = rows[j * (G + 1) + g];
        }
    };
    load_rows(threadIdx.x);
    if (threadIdx.x < G) {
        // the splits in batches of kMergeBatch whose loads all go out together
        // (a split past S reads split s0 again and weighs 0), each batch
        // raising the running reference to its largest logit
        const int g = threadIdx.x;
        float top = kNoLogit, den = 0.f;
        for (int s0 = 0; s0 < S; s0 += kMergeBatch) {
            float m[kMergeBatch], l[kMergeBatch];
#pragma unroll
            for (int i = 0; i < kMergeBatch; ++i) {
                const int s = s0 + i < S ? s0 + i : s0;
                m[i] = ml[(s * G + g) * 2];
                l[i] = ml[(s * G + g) * 2 + 1];
            }
            float bt = top;
#pragma unroll
            for (int i = 0; i < kMergeBatch; ++i) bt = fmaxf(bt, m[i]);
            if (s0 > 0) den *= __builtin_amdgcn_exp2f(top - bt);
            top = bt;
#pragma unroll
            for (int i = 0; i < kMergeBatch; ++i)
                if (s0 + i < S) den += l[i] * __builtin_amdgcn_exp2f(m[i] - top);
        }
        mg[threadIdx.x] = top;
        lg[threadIdx.x] = den;
    }
    __syncthreads();
    float M[G], Lw[G], inv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        M[g] = mg[g];
        Lw[g] = lg[g];
        inv[g] = 1.f / Lw[g];
    }
    unsigned long long best = ~0ull;
    for (int j0 = threadIdx.x; j0 < n; j0 += kRowsAtOnce * kAttnThreads) {
        if (j0 != (int)threadIdx.x) load_rows(j0);
#pragma unroll
        for (int r = 0; r < kRowsAtOnce; ++r) {
            const int j = j0 + r * kAttnThreads;
            float a = 0.f, rest = 0.f;
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float w = __builtin_amdgcn_exp2f(x[r][g] - M[g]);
                a = fmaf(w, inv[g], a);
                rest = fmaf(fmaxf(Lw[g] - w, 0.f), inv[g], rest);
            }
            const float sc = rest > 0.f ? (a / rest) * x[r][G] : __builtin_inff();  // the 1/G cancels
            const unsigned long long k = ((unsigned long long)score_key(sc) << 32) | (uint32_t)~(uint32_t)j;
            best = j < n && k < best ? k : best;
        }
    }
    best = wave_min_u64(best);
    if (lane_id() == 0) wbest[wave_id()] = best;
    __syncthreads();
    unsigned long long m = ~0ull;
#pragma unroll
    for (int q = 0; q < kAttnWaves; ++q) m = wbest[q] < m ? wbest[q] : m;
    return m;
}

// Merges a unit's splits into the attention output of its G query rows, then
// evicts (n = N + 1: the row with the lowest score, the highest slot among
// equal lowest scores; Sec. 2.1, Eq. eviction), moves row N into the freed
// slot below N (slot reuse) and updates the running sum.  Launched after the
// split kernel, so every row has been read before anything moves.
//
// The eviction is the work of LPR lanes of the last wave, lane c owning the
// columns of chunk c of a row.  Every lane of the block loads its state
// columns, its chunk of the newest row (row N when evicting) and the argmin
// words at once (lanes outside the eviction read chunk 0); only the evicted
// row's chunk waits for the argmin, and it goes out with the loads of the
// split partials, so that the block waits for memory twice.  Each lane reads
// its chunk of the evicted row before it overwrites it, so no barrier is
// needed.
template <int DT, int D, int G, bool CAOTE>
__global__ void __launch_bounds__(kAttnThreads) attn_combine_kernel(const UnitParams p) {
    using A = AttnShape<DT, D>;
    using E = Elem<DT>;
    constexpr int EPL = A::EPL, LPR = A::LPR;
    constexpr int kOut = (G * D + kAttnThreads - 1) / kAttnThreads;  // outputs per thread
    const int head = blockIdx.x;
    const int sl = blockIdx.y / p.num_layers, layer = blockIdx.y % p.num_layers;
    const int ul = (sl * p.num_layers + layer) * p.num_kv_heads + head;
    const int64_t u = (int64_t)p.unit0 + ul;
    const int n = p.nN[2 * sl], N = p.nN[2 * sl + 1];
    const int64_t off = (int64_t)sl * p.s_seq + (int64_t)layer * p.s_layer + (int64_t)head * p.s_head;
    char *kb = p.k + off;
    char *vb = p.v + off;
    const uint32_t ss32 = p.s_slot;
    double *st = p.running_sum + u * (D + 1);
    const int S = p.splits;
    const bool evict = n > N;  // the host admits n <= N + 1 only
    // The eviction lanes: the first LPR lanes of the last wave, lane c owning
    // chunk c of a row.  Every lane loads (the others chunk 0, so that no
    // loaded value leaves a branch): first what does not depend on the evicted
    // slot, then the lowest (key, ~slot), from the splits' argmin words (one
    // per lane, the minimum taken by each wave) or, for FastCAOTE, from every
    // row's score; the evicted row's chunk then goes out with the output
    // loads below.
    constexpr int kEvWave = kAttnWaves - 1;
    static_assert(LPR <= 64, "the chunks of a row fit one wave");
    const int c = threadIdx.x - kEvWave * 64;
    const bool ev = c >= 0 && c < LPR;
    const int ce = ev ? c : 0;
    const int last = n > 0 ? n - 1 : 0;
    const double cnt = st[D];
    double old[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) old[i] = st[ce * EPL + i];
    const uint4 kl = load_stream(kb, row_off(last, ss32, ce));
    const uint4 vl = load_stream(vb, row_off(last, ss32, ce));
    // row N's position (any readable word when there is none to move), by a
    // vector load (the index in VGPRs), so that no wait for it comes early
    const bool has_pos = p.pos && evict;
    const int32_t *pbase = has_pos ? p.pos : reinterpret_cast<const int32_t *>(kb);
    int64_t pix = has_pos ? u * p.capacity + N : 0;
    asm volatile("" : "+v"(pix));
    const int32_t pl = pbase[pix];
    unsigned long long lowest = ~0ull;
    if constexpr (CAOTE) {
        if (evict) lowest = caote_argmin<G>(p, u, n, p.ws_ml + u * S * G * 2, S);  // uniform branch
    } else {
        for (int s = lane_id(); s < S; s += 64) lowest = p.ws_amin[u * S + s] < lowest ? p.ws_amin[u * S + s] : lowest;
        lowest = wave_min_u64(lowest);
    }
    const int j = evict ? (int)~(uint32_t)lowest : -1;
    const uint4 xj = load_stream(vb, row_off(j >= 0 ? j : 0, ss32, ce));  // used after the outputs
    // outputs: the splits in batches of kMergeBatch whose loads all go out
    // together (a split past S reads split s0 again and weighs 0), each batch
    // raising the running reference to its largest logit
    float *orow = p.attn_out + (((int64_t)sl * p.num_layers + layer) * p.num_kv_heads + head) * G * D;
    const float *ml = p.ws_ml + u * S * G * 2;
    const float *pa = p.ws_acc + u * S * G * D;
#pragma unroll
    for (int o = 0; o < kOut; ++o) {
        const int idx = threadIdx.x + o * kAttnThreads;
        if (idx < G * D) {
            const int g = idx / D, cc = idx % D;
            float top = kNoLogit, num = 0.f, den = 0.f;
            for (int s0 = 0; s0 < S; s0 += kMergeBatch) {
                float m[kMergeBatch], l[kMergeBatch], a[kMergeBatch];
#pragma unroll
                for (int i = 0; i < kMergeBatch; ++i) {
                    const int s = s0 + i < S ? s0 + i : s0;
                    m[i] = ml[(s * G + g) * 2];
                    l[i] = ml[(s * G + g) * 2 + 1];
                    a[i] = pa[(s * G + g) * D + cc];
                }
                float bt = top;
#pragma unroll
                for (int i = 0; i < kMergeBatch; ++i) bt = fmaxf(bt, m[i]);
                if (s0 > 0) {  // the earlier batches' sums to the new reference
                    const float r = __builtin_amdgcn_exp2f(top - bt);
                    num *= r;
                    den *= r;
                }
                top = bt;
#pragma unroll
                for (int i = 0; i < kMergeBatch; ++i) {
                    const float f = s0 + i < S ? __builtin_amdgcn_exp2f(m[i] - top) : 0.f;
                    num = fmaf(a[i], f, num);
                    den = fmaf(l[i], f, den);
                }
            }
            orow[g * D + cc] = n > 0 ? num / den : 0.f;
        }
    }
    if (ev) {
        const int count = (cnt >= 0.0 && cnt <= (double)n && cnt == (double)(int)cnt) ? (int)cnt : 0;
        // the rows the state does not cover, in slot order (the newest one is loaded)
        double f[EPL];
#pragma unroll
        for (int i = 0; i < EPL; ++i) f[i] = 0.0;
        for (int r = count; r < n; ++r) {
            float x[EPL];
            E::unpack(r == last ? vl : load_stream(vb, row_off(r, ss32, c)), x);
#pragma unroll
            for (int i = 0; i < EPL; ++i) f[i] += (double)x[i];
        }
        double part[EPL];
#pragma unroll
        for (int i = 0; i < EPL; ++i) part[i] = (count > 0 ? old[i] : 0.0) + f[i];
        // the evicted row leaves the running sum; lane c read its chunk before
        // the move below overwrites it
        if (j >= 0) {
            float x[EPL];
            E::unpack(xj, x);
#pragma unroll
            for (int i = 0; i < EPL; ++i) part[i] -= (double)x[i];
        }
#pragma unroll
        for (int i = 0; i < EPL; ++i) st[c * EPL + i] = part[i];
        if (c == 0) st[D] = (double)(evict ? N : n);
        if (j >= 0 && j < N) {  // slot reuse: the newest kept row N (= n - 1) fills the hole
            store_stream(kb, row_off(j, ss32, c), kl);
            store_stream(vb, row_off(j, ss32, c), vl);
            if (p.pos && c == 0) p.pos[u * p.capacity + j] = pl;
        }
    }
}

template <int DT, int D, int G> void *attn_kernel_for(bool caote, bool combine) {
    if (caote)
        return combine ? reinterpret_cast<void *>(&attn_combine_kernel<DT, D, G, true>)
                       : reinterpret_cast<void *>(&attn_split_kernel<DT, D, G, true>);
    return combine ? reinterpret_cast<void *>(&attn_combine_kernel<DT, D, G, false>)
                   : reinterpret_cast<void *>(&attn_split_kernel<DT, D, G, false>);
}
template <int DT, int D> void *attn_kernel_for(int group, bool caote, bool combine) {
    switch (group) {
        case 1: return attn_kernel_for<DT, D, 1>(caote, combine);
        case 2: return attn_kernel_for<DT, D, 2>(caote, combine);
        case 4: return attn_kernel_for<DT, D, 4>(caote, combine);
    }
    return nullptr;
}
template <int DT> void *attn_kernel_for(int head_dim, int group, bool caote, bool combine) {
    switch (head_dim) {
        case 64: return attn_kernel_for<DT, 64>(group, caote, combine);
        case 128: return attn_kernel_for<DT, 128>(group, caote, combine);
        case 256: return attn_kernel_for<DT, 256>(group, caote, combine);
    }
    return nullptr;
}

// The ABI's variants onto the kernel's score forms (a key-side variant is the
// value-side form on the rows the host passes in V's place).
template <int DT, int D> void *step_kernel_for(int variant) {
    switch (variant) {
        case 0: case 3: return reinterpret_cast<void *>(&step_kernel<DT, D, kL2>);
        case 1: case 4: return reinterpret_cast<void *>(&step_kernel<DT, D, kDir>);
        case 2: return reinterpret_cast<void *>(&step_kernel<DT, D, kNorm>);
        case 5: return reinterpret_cast<void *>(&step_kernel<DT, D, kKeepSmallest>);
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

hipError_t launch(void *fn, int num_seqs, size_t lds_bytes, hipStream_t stream,
                  const UnitParams &p) {
    if (!fn) return hipErrorInvalidDeviceFunction;
    void *args[] = {const_cast<UnitParams *>(&p)};
    const dim3 grid(p.num_kv_heads, p.num_layers, num_seqs);
    return hipLaunchKernel(fn, grid, dim3(NT), args, lds_bytes, stream);
}

}  // namespace

hipError_t launch_step(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                       int variant, size_t lds_bytes, hipStream_t stream) {
    void *fn = dtype == 0 ? step_kernel_for<0>(head_dim, variant)
                          : step_kernel_for<1>(head_dim, variant);
    return launch(fn, num_seqs, lds_bytes, stream, p);
}

hipError_t launch_select(const UnitParams &p, int num_seqs, size_t lds_bytes,
                         hipStream_t stream) {
    return launch(reinterpret_cast<void *>(&select_kernel), num_seqs, lds_bytes, stream, p);
}

// Plain streaming read with the pass kernel's access pattern: each workgroup
// walks one contiguous part of the buffer, every lane keeping eight 16-byte
// loads in flight, and folds the data into one word, stored only if it equals
// a fixed constant.
constexpr int kReadGroups = 1024;
__global__ void __launch_bounds__(256) stream_read_kernel(const u32x4 *buf, size_t n16, uint32_t *sink) {
    constexpr int kIn = 8, kTile = kIn * 256;
    const size_t per = (n16 + kReadGroups - 1) / kReadGroups;
    const size_t b0 = (size_t)blockIdx.x * per;
    const size_t b1 = b0 + per < n16 ? b0 + per : n16;
    uint32_t x = 0u;
    size_t i = b0;
    for (; i + kTile <= b1; i += kTile) {
        u32x4 w[kIn];
#pragma unroll
        for (int k = 0; k < kIn; ++k) w[k] = __builtin_nontemporal_load(buf + i + k * 256 + threadIdx.x);
#pragma unroll
        for (int k = 0; k < kIn; ++k) x ^= w[k].x ^ w[k].y ^ w[k].z ^ w[k].w;
    }
    for (size_t j = i + threadIdx.x; j < b1; j += 256) {
        const u32x4 w = __builtin_nontemporal_load(buf + j);
        x ^= w.x ^ w.y ^ w.z ^ w.w;
    }
    if (x == 0x9E3779B9u) sink[0] = x;
}

hipError_t launch_compact(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                          size_t lds_bytes, hipStream_t stream) {
    void *fn = dtype == 0 ? compact_kernel_for<0>(head_dim) : compact_kernel_for<1>(head_dim);
    return launch(fn, num_seqs, lds_bytes, stream, p);
}

hipError_t launch_geometry(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                           size_t lds_bytes, hipStream_t stream) {
    void *fn = dtype == 0 ? geometry_kernel_for<0>(head_dim) : geometry_kernel_for<1>(head_dim);
    return launch(fn, num_seqs, lds_bytes, stream, p);
}

hipError_t launch_attn(const UnitParams &p, int num_seqs, int dtype, int head_dim, int group,
                       bool caote, size_t split_lds, hipStream_t stream) {
    void *fs = dtype == 0 ? attn_kernel_for<0>(head_dim, group, caote, false)
                          : attn_kernel_for<1>(head_dim, group, caote, false);
    void *fc = dtype == 0 ? attn_kernel_for<0>(head_dim, group, caote, true)
                          : attn_kernel_for<1>(head_dim, group, caote, true);
    if (!fs || !fc) return hipErrorInvalidDeviceFunction;
    void *args[] = {const_cast<UnitParams *>(&p)};
    const unsigned sz = (unsigned)(num_seqs * p.num_layers);
    hipError_t e = hipLaunchKernel(fs, dim3(p.splits, p.num_kv_heads, sz), dim3(kAttnThreads), args,
                                   split_lds, stream);
    if (e != hipSuccess) return e;
    return hipLaunchKernel(fc, dim3(p.num_kv_heads, sz), dim3(kAttnThreads), args, 0, stream);
}

hipError_t scratch_memory(hipStream_t stream, void **ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (stream) {  // the launch goes to the stream's device: it must be the current one
        hipDevice_t sdev = -1;
        e = hipStreamGetDevice(stream, &sdev);
        if (e != hipSuccess) return e;
        if (sdev != dev) return hipErrorInvalidDevice;
    }
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {  // once per device, with that device current
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

#if VD_DEBUG
hipError_t debug_take_error_word(unsigned int *out) {
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return e;
    unsigned int w = 0u;
    e = hipMemcpyFromSymbol(&w, HIP_SYMBOL(vd_debug_error_word), sizeof w, 0, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return e;
    const unsigned int zero = 0u;
    e = hipMemcpyToSymbol(HIP_SYMBOL(vd_debug_error_word), &zero, sizeof zero, 0, hipMemcpyHostToDevice);
    *out = w;
    return e;
}
#endif

hipError_t launch_stream_read(const void *buf, size_t n16, uint32_t *sink, hipStream_t stream) {
    hipLaunchKernelGGL(stream_read_kernel, dim3(kReadGroups), dim3(256), 0, stream,
                       reinterpret_cast<const u32x4 *>(buf), n16, sink);
    return hipGetLastError();
}

}  // namespace vd
