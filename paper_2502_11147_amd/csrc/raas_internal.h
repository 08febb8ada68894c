// Internal interface between the host runtime and the gfx950 kernels of the
// page-based RaaS decode path. Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace raas {

enum SlotState : int32_t { kFree = 0, kPinned = 1, kEvictable = 2 };

// Per-unit record: [tail slot or -1, next logical page id, clock, last evicted id]
enum UnitField : int { kTail = 0, kNextLid = 1, kClock = 2, kEvicted = 3 };

// Tokens of one attention block: two 16-row MFMA tiles.
constexpr int kBlockTokens = 32;
// Waves per attention workgroup.
constexpr int kAttnWaves = 4;
// Upper bound on attention splits per unit (sizes the partials buffer).
constexpr int kMaxSplits = 64;

// One layer of the pool, as the kernels see it. Unit u = seq * n_kv_heads + kv_head.
struct LayerView {
    void* K;         // [U][Lcap][D] in the block-swizzled (bf16) or plain (fp32) layout
    void* V;         // [U][Lcap][D] likewise
    void* kmin;      // [U][S][D] per-page per-channel key minimum, pool dtype
    void* kmax;      // [U][S][D] per-page per-channel key maximum
    int32_t* lid;    // [U][S] logical page id, -1 when free
    int32_t* ts;     // [U][S] timestamp, -1 unless evictable
    int32_t* state;  // [U][S] SlotState
    int32_t* fill;   // [U][S] tokens in the page
    int32_t* unit;   // [U][4] UnitField
    int32_t* err;    // device flag, nonzero after an internal inconsistency
    int U, G, D, ps, S, Lcap;
    int bf16;        // 1: bf16 pool, 0: fp32 pool
};

struct StepIO {
    const void* q;       // [U][G][D]
    const void* k_new;   // [U][D]
    const void* v_new;   // [U][D]
    void* out;           // [U][G][D]
    int32_t* page_table_out;
    int32_t* timestamps_out;
    int32_t* evicted_out;
};

// Launchers (asynchronous on `stream`; return the launch status).
hipError_t launch_prefill(const LayerView& L, const void* k, const void* v, int P, int keep_pages,
                          hipStream_t stream);
hipError_t launch_append(const LayerView& L, const StepIO& io, hipStream_t stream);
hipError_t launch_attention(const LayerView& L, const StepIO& io, int nsplit, int blocks_per_split,
                            float* partials, hipStream_t stream);
hipError_t launch_merge(const LayerView& L, const StepIO& io, int nsplit, const float* partials,
                        hipStream_t stream);
hipError_t launch_score(const LayerView& L, const StepIO& io, double r, hipStream_t stream);

}  // namespace raas
