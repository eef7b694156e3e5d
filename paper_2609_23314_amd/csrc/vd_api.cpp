// Host side of the C ABI declared in include/vd.h: argument validation (before
// anything touches the GPU), the per-launch LDS plan, and the launches on the
// caller's stream.  Sequences are processed in launches of at most
// kMaxSeqsPerLaunch, whose n and N travel as kernel arguments.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <utility>
#include <cstdint>
#include <cstring>

#include "vd.h"
#include "vd_debug.h"
#include "vd_launch.h"

namespace {

using vd::UnitParams;

int64_t elem_bytes(int32_t dtype) { return dtype == VD_DTYPE_BF16 ? 2 : 4; }
int64_t align16(int64_t x) { return (x + 15) & ~int64_t(15); }
bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

vd_status check_desc(const vd_cache_desc *d) {
    if (!d || !d->v) return VD_ERR_INVALID_ARG;
    if (d->dtype != VD_DTYPE_BF16 && d->dtype != VD_DTYPE_F32) return VD_ERR_INVALID_ARG;
    if (d->num_seqs < 1 || d->num_layers < 1 || d->num_kv_heads < 1 || d->num_q_heads < 1)
        return VD_ERR_INVALID_ARG;
    if (d->num_q_heads % d->num_kv_heads != 0) return VD_ERR_INVALID_ARG;
    if (d->head_dim < 1 || d->capacity < 1) return VD_ERR_INVALID_ARG;
    if (d->head_dim != 64 && d->head_dim != 128 && d->head_dim != 256) return VD_ERR_UNSUPPORTED;
    if (d->capacity > VD_MAX_CAPACITY) return VD_ERR_UNSUPPORTED;
    if (d->stride_seq < 0 || d->stride_layer < 0 || d->stride_head < 0 || d->stride_slot < 0)
        return VD_ERR_INVALID_ARG;
    if (d->stride_slot < d->head_dim) return VD_ERR_INVALID_ARG;  // rows would overlap
    if (d->num_layers > 65535) return VD_ERR_UNSUPPORTED;  // one grid row per layer
    const int64_t units = int64_t(d->num_seqs) * d->num_layers * d->num_kv_heads;
    if (units > INT32_MAX || units * int64_t(d->capacity) > (int64_t(1) << 47))
        return VD_ERR_UNSUPPORTED;
    const int64_t es = elem_bytes(d->dtype);
    // a unit's slab is addressed with 32-bit byte offsets
    if (int64_t(d->capacity) * d->stride_slot * es > int64_t(UINT32_MAX)) return VD_ERR_UNSUPPORTED;
    const int64_t strides[4] = {d->stride_seq, d->stride_layer, d->stride_head, d->stride_slot};
    for (int64_t s : strides)
        if ((s * es) % 16 != 0) return VD_ERR_INVALID_ARG;  // every row 16-byte aligned
    if (!aligned(d->v, 16) || (d->k && !aligned(d->k, 16))) return VD_ERR_INVALID_ARG;
    if (d->k && d->k == d->v) return VD_ERR_INVALID_ARG;
    return VD_OK;
}

vd_status check_counts(const vd_cache_desc *d, const int32_t *n_valid, const int32_t *budget) {
    if (!n_valid) return VD_ERR_INVALID_ARG;
    for (int s = 0; s < d->num_seqs; ++s) {
        if (n_valid[s] < 0 || n_valid[s] > d->capacity) return VD_ERR_INVALID_ARG;
        if (budget && budget[s] < 1) return VD_ERR_INVALID_ARG;
    }
    return VD_OK;
}

UnitParams base_params(const vd_cache_desc *d, int s0, int ns, const int32_t *n_valid,
                       const int32_t *budget) {
    UnitParams p;
    std::memset(&p, 0, sizeof p);
    const int64_t es = elem_bytes(d->dtype);
    p.k = d->k ? static_cast<char *>(d->k) + int64_t(s0) * d->stride_seq * es : nullptr;
    p.v = static_cast<char *>(d->v) + int64_t(s0) * d->stride_seq * es;
    p.s_seq = d->stride_seq * es;
    p.s_layer = d->stride_layer * es;
    p.s_head = d->stride_head * es;
    p.s_slot = uint32_t(d->stride_slot * es);
    p.num_layers = d->num_layers;
    p.num_kv_heads = d->num_kv_heads;
    p.unit0 = s0 * d->num_layers * d->num_kv_heads;
    p.capacity = d->capacity;
    for (int i = 0; i < ns; ++i) {
        p.nN[2 * i] = n_valid[s0 + i];
        p.nN[2 * i + 1] = budget ? budget[s0 + i] : INT32_MAX;
    }
    return p;
}

// Key-side scores take the same forms on the key rows: the kernel scores the
// rows it is handed as V (and sums them into the running sum) and moves the
// other tensor alongside, so for those the host hands it K in V's place.
bool key_side(vd_variant variant) {
    return variant == VD_SCORE_KEY_L2 || variant == VD_SCORE_KEY_DIR || variant == VD_SCORE_KEY_NORM;
}
bool pass_variant(vd_variant variant) { return variant >= VD_SCORE_L2 && variant <= VD_SCORE_KEY_NORM; }
void hand_scored_rows(UnitParams &p, vd_variant variant) {
    if (key_side(variant)) std::swap(p.k, p.v);
}

// Plans the dynamic LDS of the pass kernel for one launch.
vd_status plan_step_lds(const vd_cache_desc *d, UnitParams &p, int ns, bool score_mode,
                        bool have_state, bool want_scores, size_t &lds_bytes) {
    const int64_t row_bytes = int64_t(d->head_dim) * elem_bytes(d->dtype);
    int nmax = 0, keys_cap = 0, evict_cap = 0, move_cap = 0, want_rows = 0;
    for (int i = 0; i < ns; ++i) {
        const int n = p.nN[2 * i], N = p.nN[2 * i + 1];
        nmax = std::max(nmax, n);
        if (want_scores) keys_cap = std::max(keys_cap, n);  // scores leave through LDS
        if (!score_mode && n > N) {
            keys_cap = std::max(keys_cap, n);
            evict_cap = std::max(evict_cap, n - N);
            move_cap = std::max(move_cap, std::min(N, n - N));
            want_rows = std::max(want_rows, have_state ? n - N : n);
        } else if (!have_state) {
            want_rows = std::max(want_rows, n);
        }
    }
    // keys, then (when the unit selects) the second histogram buffer; the fp64
    // reduction scratch aliases the region
    const int64_t red_bytes = int64_t(vd::kWaves) * d->head_dim * 8;
    const int64_t sel_bytes = keys_cap > 0 ? align16(int64_t(keys_cap) * 4) + int64_t(vd::kBins) * 4 : 0;
    const int64_t keys_bytes = align16(std::max<int64_t>(sel_bytes, red_bytes));
    const int64_t lists_bytes = align16(int64_t(evict_cap + move_cap) * 4);
    const int64_t used = int64_t(sizeof(vd::LdsHead)) + keys_bytes + lists_bytes;
    if (used > vd::kLdsBytes) return VD_ERR_UNSUPPORTED;
    // as many of the rows to stage as fit (the kernel streams the rest twice)
    const int64_t stash_rows = std::min<int64_t>(want_rows, (vd::kLdsBytes - used) / row_bytes);
    p.off_keys = int32_t(sizeof(vd::LdsHead));
    p.off_lists = int32_t(p.off_keys + keys_bytes);
    p.off_stash = int32_t(p.off_lists + lists_bytes);
    p.keys_cap = keys_cap;
    p.evict_cap = evict_cap;
    p.move_cap = move_cap;
    p.stash_rows = int32_t(stash_rows);
    lds_bytes = size_t(used + stash_rows * row_bytes);
    return VD_OK;
}

vd_status launched(hipError_t e) { return e == hipSuccess ? VD_OK : VD_ERR_HIP; }

// Row splits of the fused decode attention: about 768 workgroups of 256
// threads over the whole launch (three per CU, what stays resident at the
// split kernel's register use; more splits were measured slower), each split
// a whole number of the split kernel's two-row tiles.  FastCAOTE keeps every
// row's logits and distance of a split in LDS until the split ends, so its
// splits hold at most kCaoteSplitRows rows.
constexpr int kCaoteSplitRows = 2048;
struct AttnPlan {
    int group, splits, rows, groups;
    int64_t units;
};
AttnPlan attn_plan(const vd_cache_desc *d, vd_variant variant) {
    AttnPlan a;
    a.group = d->num_q_heads / d->num_kv_heads;
    a.units = int64_t(d->num_seqs) * d->num_layers * d->num_kv_heads;
    const int lpr = int(d->head_dim * elem_bytes(d->dtype) / 16);
    a.groups = (vd::kAttnThreads / 64) * (64 / lpr);
    const int tile = 2 * a.groups;
    int64_t want = std::min<int64_t>(64, std::max<int64_t>(1, (768 + a.units - 1) / a.units));
    if (variant == VD_SCORE_FASTCAOTE)
        want = std::max<int64_t>(want, (d->capacity + kCaoteSplitRows - 1) / kCaoteSplitRows);
    int rows = int((d->capacity + want - 1) / want);
    rows = (rows + tile - 1) / tile * tile;
    if (variant == VD_SCORE_FASTCAOTE) rows = std::min(rows, kCaoteSplitRows);
    a.rows = rows;
    a.splits = (d->capacity + rows - 1) / rows;
    return a;
}
// Workspace: partial outputs, then (max, sum) pairs, then the argmin words,
// then (FastCAOTE) the G logits and the distance of every row of every unit.
struct AttnWs {
    int64_t acc, ml, amin, rows, total;  // byte offsets and the total
};
AttnWs attn_ws_layout(const vd_cache_desc *d, const AttnPlan &a, vd_variant variant) {
    const int64_t parts = a.units * a.splits;
    AttnWs w;
    w.acc = 0;
    w.ml = align16(parts * a.group * d->head_dim * 4);
    w.amin = w.ml + align16(parts * a.group * 2 * 4);
    w.rows = w.amin + align16(parts * 8);
    w.total = w.rows + (variant == VD_SCORE_FASTCAOTE
                            ? align16(a.units * int64_t(d->capacity) * (a.group + 1) * 4) : 0);
    return w;
}

// Validation shared by the fused decode step's entry points (host only, no
// HIP call); on success `plan` and `ws` describe the launch.
vd_status check_decode(const vd_cache_desc *desc, const float *q, float scale,
                       const int32_t *n_valid, const int32_t *budget, vd_variant variant,
                       const double *running_sum, const int32_t *pos, const float *out,
                       AttnPlan &plan, AttnWs &ws) {
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if (!desc->k) return VD_ERR_INVALID_ARG;
    if (!budget) return VD_ERR_INVALID_ARG;
    if ((st = check_counts(desc, n_valid, budget)) != VD_OK) return st;
    if (variant != VD_SCORE_L2 && variant != VD_SCORE_FASTCAOTE) return VD_ERR_INVALID_ARG;
    const int group = desc->num_q_heads / desc->num_kv_heads;
    if (group != 1 && group != 2 && group != 4) return VD_ERR_UNSUPPORTED;
    for (int s = 0; s < desc->num_seqs; ++s)
        if (n_valid[s] - 1 > budget[s]) return VD_ERR_UNSUPPORTED;  // one token evicted at most
    if (!q || !out || !aligned(q, 4) || !aligned(out, 4)) return VD_ERR_INVALID_ARG;
    if (!running_sum || !aligned(running_sum, 8) || (pos && !aligned(pos, 4)))
        return VD_ERR_INVALID_ARG;
    if (!std::isfinite(scale)) return VD_ERR_INVALID_ARG;
    plan = attn_plan(desc, variant);
    ws = attn_ws_layout(desc, plan, variant);
    return VD_OK;
}

// Launches of the fused decode step on a validated call, with the workspace
// at `wsp` (ws.total bytes, 16-byte aligned).
vd_status launch_decode(const vd_cache_desc *desc, const float *q, float scale,
                        const int32_t *n_valid, const int32_t *budget, vd_variant variant,
                        double *running_sum, int32_t *pos, float *out, const AttnPlan &a,
                        const AttnWs &ws, char *wsp, hipStream_t stream) {
    const int D = desc->head_dim, L = desc->num_layers, group = a.group;
    float *ws_acc = reinterpret_cast<float *>(wsp + ws.acc);
    float *ws_ml = reinterpret_cast<float *>(wsp + ws.ml);
    auto *ws_amin = reinterpret_cast<unsigned long long *>(wsp + ws.amin);
    const bool caote = variant == VD_SCORE_FASTCAOTE;
    float *ws_rows = caote ? reinterpret_cast<float *>(wsp + ws.rows) : nullptr;
    const int seqs_per_launch = std::max(1, std::min(vd::kMaxSeqsPerLaunch, 65535 / L));
    const int64_t row_floats = int64_t(L) * desc->num_q_heads * D;  // q / out floats per sequence
    const size_t split_lds = size_t(2 * D) * 4 + size_t(2 * a.groups * group) * 4 +
                             size_t(vd::kAttnThreads / 64) * 8 + size_t(group) * a.groups * D * 4 +
                             (caote ? size_t(a.rows) * (group + 1) * 4 : 0);
    for (int s0 = 0; s0 < desc->num_seqs; s0 += seqs_per_launch) {
        const int ns = std::min(seqs_per_launch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, budget);
        p.running_sum = running_sum;
        p.pos = pos;
        p.q = q + s0 * row_floats;
        p.attn_out = out + s0 * row_floats;
        p.ws_acc = ws_acc;
        p.ws_ml = ws_ml;
        p.ws_amin = ws_amin;
        p.ws_rows = ws_rows;
        p.splits = a.splits;
        p.split_rows = a.rows;
        p.qscale = float(double(scale) * 1.4426950408889634);  // log2(e)
        const vd_status st = launched(vd::launch_attn(p, ns, desc->dtype, D, group, caote, split_lds,
                                                      stream));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

}  // namespace

extern "C" {

vd_status vd_score(const vd_cache_desc *desc, const int32_t *n_valid, vd_variant variant,
                   float *scores, float *mean_out, vd_stream stream) {
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if ((st = check_counts(desc, n_valid, nullptr)) != VD_OK) return st;
    if (!pass_variant(variant)) return VD_ERR_INVALID_ARG;
    if (key_side(variant) && !desc->k) return VD_ERR_INVALID_ARG;
    if (!scores || !aligned(scores, 4) || (mean_out && !aligned(mean_out, 4)))
        return VD_ERR_INVALID_ARG;
    for (int s0 = 0; s0 < desc->num_seqs; s0 += vd::kMaxSeqsPerLaunch) {
        const int ns = std::min(vd::kMaxSeqsPerLaunch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, nullptr);
        hand_scored_rows(p, variant);
        p.mode = vd::kModeScore;
        p.scores = scores;
        p.mean_out = mean_out;
        size_t lds = 0;
        if ((st = plan_step_lds(desc, p, ns, true, false, true, lds)) != VD_OK) return st;
        st = launched(vd::launch_step(p, ns, desc->dtype, desc->head_dim, variant, lds,
                                      reinterpret_cast<hipStream_t>(stream)));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

vd_status vd_select_topn(const vd_cache_desc *desc, const float *scores, const int32_t *n_valid,
                         const int32_t *budget, uint8_t *keep_mask, vd_stream stream) {
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if (!budget) return VD_ERR_INVALID_ARG;
    if ((st = check_counts(desc, n_valid, budget)) != VD_OK) return st;
    if (!scores || !keep_mask || !aligned(scores, 4)) return VD_ERR_INVALID_ARG;
    for (int s0 = 0; s0 < desc->num_seqs; s0 += vd::kMaxSeqsPerLaunch) {
        const int ns = std::min(vd::kMaxSeqsPerLaunch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, budget);
        p.scores_in = scores;
        p.keep = keep_mask;
        int nmax = 0;
        for (int i = 0; i < ns; ++i) nmax = std::max(nmax, p.nN[2 * i]);
        p.off_keys = int32_t(sizeof(vd::LdsHead));
        p.keys_cap = nmax;
        const size_t lds = sizeof(vd::LdsHead) + size_t(align16(int64_t(nmax) * 4)) + size_t(vd::kBins) * 4;
        p.off_lists = int32_t(lds);  // the end of the keys region (keys, then the second histogram)
        if (lds > size_t(vd::kLdsBytes)) return VD_ERR_UNSUPPORTED;
        st = launched(vd::launch_select(p, ns, lds, reinterpret_cast<hipStream_t>(stream)));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

vd_status vd_compact(const vd_cache_desc *desc, const uint8_t *keep_mask, const int32_t *n_valid,
                     const int32_t *budget, int32_t *pos, vd_stream stream) {
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if (!budget) return VD_ERR_INVALID_ARG;
    if ((st = check_counts(desc, n_valid, budget)) != VD_OK) return st;
    if (!keep_mask || (pos && !aligned(pos, 4))) return VD_ERR_INVALID_ARG;
    for (int s0 = 0; s0 < desc->num_seqs; s0 += vd::kMaxSeqsPerLaunch) {
        const int ns = std::min(vd::kMaxSeqsPerLaunch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, budget);
        p.keep_in = keep_mask;
        p.pos = pos;
        int holes = 0, movers = 0;
        for (int i = 0; i < ns; ++i) {
            const int n = p.nN[2 * i], N = p.nN[2 * i + 1];
            if (n > N) {
                holes = std::max(holes, std::min(N, n));
                movers = std::max(movers, n - N);
            }
        }
        if (holes == 0) continue;  // nothing exceeds its budget in this launch
        p.off_lists = int32_t(sizeof(vd::LdsHead));
        p.evict_cap = holes;
        p.move_cap = movers;
        const size_t lds = sizeof(vd::LdsHead) + size_t(align16(int64_t(holes + movers) * 4));
        if (lds > size_t(vd::kLdsBytes)) return VD_ERR_UNSUPPORTED;
        st = launched(vd::launch_compact(p, ns, desc->dtype, desc->head_dim, lds,
                                         reinterpret_cast<hipStream_t>(stream)));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

vd_status vd_evict_step(const vd_cache_desc *desc, const int32_t *n_valid, const int32_t *budget,
                        vd_variant variant, double *running_sum, int32_t *pos, float *scores_out,
                        uint8_t *keep_out, void *workspace, size_t workspace_bytes,
                        vd_stream stream) {
    (void)workspace;
    (void)workspace_bytes;
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if (!budget) return VD_ERR_INVALID_ARG;
    if ((st = check_counts(desc, n_valid, budget)) != VD_OK) return st;
    if (!pass_variant(variant)) return VD_ERR_INVALID_ARG;
    if (key_side(variant) && !desc->k) return VD_ERR_INVALID_ARG;
    if ((running_sum && !aligned(running_sum, 8)) || (pos && !aligned(pos, 4)) ||
        (scores_out && !aligned(scores_out, 4)))
        return VD_ERR_INVALID_ARG;
    for (int s0 = 0; s0 < desc->num_seqs; s0 += vd::kMaxSeqsPerLaunch) {
        const int ns = std::min(vd::kMaxSeqsPerLaunch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, budget);
        hand_scored_rows(p, variant);
        p.mode = vd::kModeStep;
        p.running_sum = running_sum;
        p.pos = pos;
        p.scores = scores_out;
        p.keep = keep_out;
        size_t lds = 0;
        if ((st = plan_step_lds(desc, p, ns, false, running_sum != nullptr, scores_out != nullptr,
                                lds)) != VD_OK)
            return st;
        st = launched(vd::launch_step(p, ns, desc->dtype, desc->head_dim, variant, lds,
                                      reinterpret_cast<hipStream_t>(stream)));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

vd_status vd_geometry(const vd_cache_desc *desc, const int32_t *n_valid, const double *k_sum,
                      const double *v_sum, double *out, vd_stream stream) {
    vd_status st = check_desc(desc);
    if (st != VD_OK) return st;
    if (!desc->k) return VD_ERR_INVALID_ARG;
    if ((st = check_counts(desc, n_valid, nullptr)) != VD_OK) return st;
    if (!out || !aligned(out, 8)) return VD_ERR_INVALID_ARG;
    if (!k_sum != !v_sum) return VD_ERR_INVALID_ARG;  // both or neither
    if ((k_sum && !aligned(k_sum, 8)) || (v_sum && !aligned(v_sum, 8))) return VD_ERR_INVALID_ARG;
    // fp64 reduction scratch, then the four centroid arrays (K hi, K lo, V hi, V lo)
    const int64_t red_bytes = int64_t(vd::kWaves) * desc->head_dim * 8;
    const int64_t ctr_bytes = int64_t(4) * desc->head_dim * 4;
    for (int s0 = 0; s0 < desc->num_seqs; s0 += vd::kMaxSeqsPerLaunch) {
        const int ns = std::min(vd::kMaxSeqsPerLaunch, desc->num_seqs - s0);
        UnitParams p = base_params(desc, s0, ns, n_valid, nullptr);
        p.geom_out = out;
        p.k_sum = k_sum;
        p.v_sum = v_sum;
        p.off_keys = int32_t(sizeof(vd::LdsHead));
        p.off_lists = int32_t(p.off_keys + red_bytes);
        const size_t lds = size_t(p.off_lists + ctr_bytes);
        st = launched(vd::launch_geometry(p, ns, desc->dtype, desc->head_dim, lds,
                                          reinterpret_cast<hipStream_t>(stream)));
        if (st != VD_OK) return st;
    }
    return VD_OK;
}

size_t vd_decode_attention_workspace_size(const vd_cache_desc *desc, vd_variant variant) {
    if (check_desc(desc) != VD_OK) return 0;
    if (variant != VD_SCORE_L2 && variant != VD_SCORE_FASTCAOTE) return 0;
    return size_t(attn_ws_layout(desc, attn_plan(desc, variant), variant).total);
}

vd_status vd_decode_attention_evict(const vd_cache_desc *desc, const float *q, float scale,
                                    const int32_t *n_valid, const int32_t *budget,
                                    vd_variant variant, double *running_sum, int32_t *pos,
                                    float *out, void *workspace, size_t workspace_bytes,
                                    vd_stream stream) {
    AttnPlan a;
    AttnWs ws;
    const vd_status st = check_decode(desc, q, scale, n_valid, budget, variant, running_sum, pos,
                                      out, a, ws);
    if (st != VD_OK) return st;
    if (!workspace || !aligned(workspace, 16)) return VD_ERR_WORKSPACE;
    if (int64_t(workspace_bytes) < ws.total) return VD_ERR_WORKSPACE;
    return launch_decode(desc, q, scale, n_valid, budget, variant, running_sum, pos, out, a, ws,
                         static_cast<char *>(workspace), reinterpret_cast<hipStream_t>(stream));
}

vd_status vd_decode_attention_evict_noalloc(const vd_cache_desc *desc, const float *q, float scale,
                                            const int32_t *n_valid, const int32_t *budget,
                                            vd_variant variant, double *running_sum, int32_t *pos,
                                            float *out, vd_stream stream) {
    AttnPlan a;
    AttnWs ws;
    const vd_status st = check_decode(desc, q, scale, n_valid, budget, variant, running_sum, pos,
                                      out, a, ws);
    if (st != VD_OK) return st;
    if (ws.total > int64_t(vd::kScratchBytes)) return VD_ERR_WORKSPACE;  // beyond the static scratch
    void *scratch = nullptr;
    const hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    if (vd::scratch_memory(hs, &scratch) != hipSuccess) return VD_ERR_HIP;
    return launch_decode(desc, q, scale, n_valid, budget, variant, running_sum, pos, out, a, ws,
                         static_cast<char *>(scratch), hs);
}

size_t vd_decode_attention_noalloc_max_bytes(void) { return vd::kScratchBytes; }

size_t vd_evict_step_workspace_size(const vd_cache_desc *desc) {
    (void)desc;
    return 0;
}

vd_status vd_stream_read(const void *buf, size_t bytes, uint32_t *sink, vd_stream stream) {
    if (!buf || !sink || bytes == 0 || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0)
        return VD_ERR_INVALID_ARG;
    return vd::launch_stream_read(buf, bytes / 16, sink, reinterpret_cast<hipStream_t>(stream)) == hipSuccess
               ? VD_OK : VD_ERR_HIP;
}

#if VD_DEBUG
vd_status vd_debug_take_error_word(uint32_t *word) {
    if (!word) return VD_ERR_INVALID_ARG;
    unsigned int w = 0u;
    if (vd::debug_take_error_word(&w) != hipSuccess) return VD_ERR_HIP;
    *word = w;
    return VD_OK;
}
#endif

const char *vd_status_string(vd_status status) {
    switch (status) {
        case VD_OK: return "ok";
        case VD_ERR_INVALID_ARG: return "invalid argument";
        case VD_ERR_UNSUPPORTED: return "unsupported shape";
        case VD_ERR_WORKSPACE: return "workspace missing or too small";
        case VD_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

}  // extern "C"
