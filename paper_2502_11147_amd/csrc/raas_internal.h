// Internal interface between the host runtime and the gfx950 kernels of the
// page-based RaaS decode path. Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace raas {

enum SlotState : int32_t { kFree = 0, kPinned = 1, kEvictable = 2 };

// Per-unit record, kUnitFields int32 each:
//  tail      slot of the page receiving decode tokens, or -1
//  next_lid  logical id the next fresh page gets
//  clock     absolute position of the next token
//  evicted   logical id evicted by the last step, or -1
//  next_slot slot the next token goes to (the tail, or the lowest free slot)
//  next_fill its position in that page (0: the page is opened by that token)
//  pinned    number of pinned prefill pages (slots 0 .. pinned-1)
enum UnitField : int { kTail = 0, kNextLid = 1, kClock = 2, kEvicted = 3, kNextSlot = 4, kNextFill = 5, kPinnedPages = 6 };
constexpr int kUnitFields = 8;

// Tokens of one attention block: two 16-row MFMA tiles.
constexpr int kBlockTokens = 32;
// Upper bound on attention splits per unit (sizes the partials buffer).
constexpr int kMaxSplits = 64;
// Dynamic LDS a step workgroup may use (gfx950 has 160 KiB per workgroup).
constexpr size_t kMaxLds = 144 * 1024;

// One layer of the pool, as the kernels see it. Unit u = seq * n_kv_heads + kv_head.
struct LayerView {
    void* K;         // [U][Lcap][D] block-swizzled (bf16) or plain (fp32)
    void* V;         // [U][Lcap][D] likewise
    void* kmin;      // [U][S][D] per-page per-channel key minimum, pool dtype
    void* kmax;      // [U][S][D] per-page per-channel key maximum
    int32_t* lid;    // [U][S] logical page id, -1 when free
    int32_t* ts;     // [U][S] timestamp, -1 unless evictable
    int32_t* state;  // [U][S] SlotState
    int32_t* fill;   // [U][S] tokens in the page
    int32_t* unit;   // [U][kUnitFields]
    int32_t* err;    // device flag, nonzero after an internal inconsistency
    double* score;   // split path: [U][S] page scores; [U][S][G] per-head bounds when agg == 1
    float* part;     // [U][nsplit][G][D+2] partial attention (split path)
    int U, G, D, ps, S, Lcap;
    int nsplit, bps;  // attention splits per unit, 32-token blocks per split
    int rev;          // 1: this step visits blocks and page groups in descending order
    int bf16;         // 1: bf16 pool, 0: fp32 pool
    int agg;          // head aggregation of the page score: 0 max, 1 sum of per-head softmax
    int rank_pinned;  // 1: pinned pages are scored and ranked (never refreshed)
    int hgrp;         // units per retention decision: 1, or n_kv_heads (units seq*hgrp .. +hgrp-1)
    int nkv;          // KV heads per sequence: unit u belongs to sequence u / nkv
    int nblk;         // 32-token blocks a step visits (from row 0): every resident row lies below
    int dbase;        // first slot decode pages may take (the prompt region's size; 0 without one)
    int pcap;         // most prompt pages kept: S-1, or the prompt region's slots
    int topk;         // prompt pages attended per step (Quest on the prompt), -1: all
    int32_t* fill_att;  // [U][S] fills the attention sees: fill, or (topk >= 0) 0 for unchosen prompt pages
    int32_t* blist;     // [U][lcap_blk] blocks a step visits (topk >= 0): chosen prompt blocks, decode blocks
    int32_t* bcnt;      // [U][2] prompt blocks and all blocks in blist
    float* pivl;        // [2][U][dbase] prompt pages' bound intervals (lower, upper) from k_prompt_intervals
    int pchunk;         // prompt pages per k_prompt_intervals workgroup; 0: the selection kernel bounds them itself
    int lcap_blk;       // Lcap / 32
    int nt;             // 1: K/V blocks streamed with non-temporal loads
    int det;            // 1: each wavefront takes a fixed interleave of the blocks (reproducible sums)
    int early;          // 1: the first score pass's loads go out before the first block is attended
};

// Prefill input of one layer: `stride` token rows per unit; per-sequence
// lengths (lens, device [batch]) or one length P; an optional device mask
// [batch] of the sequences to (re)initialise.
struct PrefillIn {
    const int32_t* lens;
    const int32_t* mask;
    int P, stride;
};

struct StepIO {
    const void* q;       // [U][G][D]
    const void* k_new;   // [U][D]
    const void* v_new;   // [U][D]
    void* out;           // [U][G][D]
    int32_t* page_table_out;
    int32_t* timestamps_out;
    int32_t* evicted_out;
    const int32_t* active;  // device [batch]: nonzero = the sequence takes this step; NULL = all
};

// Launch plan of one decode step.
struct StepPlan {
    int waves;       // wavefronts per step workgroup (bf16)
    int nsplit, bps; // splits per unit and blocks per split
    bool fused;      // true: the step workgroup also runs the epilogue (nsplit == 1, bf16)
    bool select_in_step;  // true: the step kernel chooses the prompt pages (no selection kernel)
    size_t lds;      // dynamic LDS of the step kernel
};

// work_blocks: 32-token blocks a unit's step attends (Lcap / 32 less the
// unchosen prompt blocks); grouped: retention decided per group of units, by
// the epilogue kernel;
// list_ints: LDS ints of a block list or of the in-step prompt selection (0
// without a prompt region)
StepPlan plan_step(int U, int G, int D, int S, int Lcap, int ps, int work_blocks, bool bf16, int agg,
                   bool grouped, int list_ints, int split_override,
                   int npr);
// Quest on the prompt pages: the attended fills and the block list of a step.
hipError_t launch_prompt_select(const LayerView& L, const StepIO& io, hipStream_t stream);
// Lets the step kernels use more than the default dynamic LDS.
hipError_t allow_large_lds();

// Launchers (asynchronous on `stream`; return the launch status).
// max_tok: the most tokens any selected unit keeps (min(P, kept pages * ps)).
hipError_t launch_prefill(const LayerView& L, const void* k, const void* v, const PrefillIn& in, int max_tok,
                          hipStream_t stream);
// The step kernel: attention, page scores, append; plus the epilogue when fused.
hipError_t launch_step(const LayerView& L, const StepIO& io, const StepPlan& plan, double r,
                       hipStream_t stream);
// The epilogue kernel of the split path: merge, refresh, evict, state out;
// one workgroup per group of L.hgrp units.
hipError_t launch_epilogue(const LayerView& L, const StepIO& io, double r, hipStream_t stream);

}  // namespace raas
