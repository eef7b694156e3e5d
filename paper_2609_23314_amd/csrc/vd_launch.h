// Internal contract between the host entry points (vd_api.cpp) and the
// kernels (vd_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vd {

constexpr int kBlock = 1024;              // threads per workgroup (16 waves of 64)
constexpr int kWaves = kBlock / 64;
constexpr int kMaxSeqsPerLaunch = 256;    // per-sequence n and N travel as kernel arguments
constexpr int kLdsBytes = 160 * 1024;     // LDS of one gfx950 workgroup

enum Mode : int32_t { kModeStep = 0, kModeScore = 1 };

// Fixed head of the dynamic LDS of every kernel.
constexpr int kBins = 1024;                // histogram bins of the selection
constexpr int kCand = 64;                  // candidates ranked directly by one wave

struct LdsHead {
    uint32_t bc[128];     // broadcast slots and per-wave partials
    uint32_t hist[kBins]; // selection histogram
    uint32_t cand_key[kCand];
    uint32_t cand_idx[kCand];
    float mean[256];      // fp32 mean used for scoring (its high part for L2)
    float aux[256];       // L2: the low part of the mean (mean - high part);
                          // Dir: mean / ||mean||
    double sum[256];      // fp64 column sums of all n rows
    double old_sum[256];  // fp64 column sums of the rows the state covered
};
static_assert(sizeof(LdsHead) % 16 == 0, "LDS head must keep 16-byte alignment");

// Kernel arguments.  The fields every workgroup needs before its first row
// load come first, so that one batch of scalar loads fetches them; the unit's
// (sequence, layer, head) is the workgroup's (z, y, x) position in the grid.
struct UnitParams {
    char *k;                  // first unit of the launch's first sequence; may be null
    char *v;
    double *running_sum;      // [U][D+1] or null
    int64_t s_seq, s_layer, s_head;   // strides in BYTES
    uint32_t s_slot;          // bytes from one slot to the next (a slab spans < 4 GiB)
    int32_t num_layers, num_kv_heads;
    int32_t unit0;            // global index of the launch's first unit
    int32_t capacity;
    int32_t mode;             // Mode
    int32_t stash_rows;       // rows the stash holds
    // dynamic LDS layout (byte offsets from the start of dynamic LDS)
    int32_t off_keys;         // keys, then the second histogram buffer / fp64 reduction scratch
    int32_t off_lists;        // evicted (or hole) list, then mover list
    int32_t off_stash;        // staged rows
    int32_t keys_cap;         // entries in the keys region
    int32_t evict_cap;        // entries of the first list
    int32_t move_cap;         // entries of the second list
    int32_t pad0;
    int32_t *pos;             // [U][capacity] or null
    float *scores;            // [U][capacity] or null (required in kModeScore)
    const float *scores_in;   // select kernel input
    uint8_t *keep;            // [U][capacity] or null (output of step/select)
    const uint8_t *keep_in;   // compact kernel input
    float *mean_out;          // [U][D] or null
    double *geom_out;         // [U][5] (geometry kernel)
    const double *k_sum;      // geometry: [U][D+1] column sums of K and their row count, or null
    const double *v_sum;      // geometry: the same for V, or null
    // fused decode attention
    const float *q;           // [S][L][Hq][D] of the launch's first sequence
    float *attn_out;          // [S][L][Hq][D]
    float *ws_acc;            // [U][splits][G][D] partial outputs (unnormalised)
    float *ws_ml;             // [U][splits][G][2] partial max logit (log2 units) and weight sum
    unsigned long long *ws_amin;  // [U][splits] (key << 32 | ~slot) of the lowest score
    float *ws_rows;           // FastCAOTE: [U][capacity][G + 1] log2 logits of the G heads, distance
    int32_t splits, split_rows;   // row splits per unit and rows per split
    float qscale;             // softmax scale times log2(e)
    int32_t pad1;
    int32_t nN[2 * kMaxSeqsPerLaunch];   // n and N of each sequence of the launch, interleaved
};

// Each launches one workgroup per unit of `num_seqs` sequences.
hipError_t launch_step(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                       int variant, size_t lds_bytes, hipStream_t stream);
hipError_t launch_select(const UnitParams &p, int num_seqs, size_t lds_bytes,
                         hipStream_t stream);
hipError_t launch_compact(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                          size_t lds_bytes, hipStream_t stream);
// Fused decode attention: split kernel (grid splits x heads x seqs*layers),
// then the combine kernel (grid heads x seqs*layers); G = query heads per KV head.
constexpr int kAttnThreads = 256;
hipError_t launch_attn(const UnitParams &p, int num_seqs, int dtype, int head_dim, int group,
                       bool caote, size_t split_lds, hipStream_t stream);
hipError_t launch_geometry(const UnitParams &p, int num_seqs, int dtype, int head_dim,
                           size_t lds_bytes, hipStream_t stream);
// Static device scratch of the allocation-free fused decode step (one copy per
// GPU): its size, and its address on the current device, which must be the
// device of `stream` (looked up once per device, then cached).
constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;
hipError_t scratch_memory(hipStream_t stream, void **ptr);
// Debug builds (VD_DEBUG=1): waits for the device, then returns and clears the
// word in which the kernels' LDS index checks set one bit per failing site.
hipError_t debug_take_error_word(unsigned int *out);
// Reads n16 16-byte words once over the whole GPU (a measurement aid).
hipError_t launch_stream_read(const void *buf, size_t n16, uint32_t *sink, hipStream_t stream);

}  // namespace vd
