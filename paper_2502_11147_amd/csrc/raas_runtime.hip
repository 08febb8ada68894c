// Host runtime of the page-based RaaS decode path: argument validation, the
// fixed HBM page pool, and the per-step launch sequence on the caller's
// stream. Implements include/raas.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "raas.h"
#include "raas_internal.h"

using namespace raas;

namespace {

thread_local std::string g_last_error;

raas_status fail(raas_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
raas_status fail(raas_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

raas_status hip_fail(hipError_t e, const char* what) {
    return fail(RAAS_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kKernels = 3;  // step kernel, epilogue kernel, prompt selection kernel
constexpr size_t kProfRing = 8192;

struct Timing {
    std::vector<hipEvent_t> start, stop;  // ring of recorded pairs
    size_t head = 0, count = 0;           // pairs recorded since the last read
    double folded_ms = 0.0;               // time of pairs recycled before the read
    int64_t folded_n = 0;
    bool started = false;                 // the open pair's start event was recorded
};

}  // namespace

struct raas_pool {
    raas_config cfg;
    int U, G, D, ps, S, Lcap, esz;
    size_t kv_layer_elems, meta_layer_elems, rep_layer_elems;
    void* K = nullptr;
    void* V = nullptr;
    void* kmin = nullptr;
    void* kmax = nullptr;
    int32_t* meta = nullptr;  // lid, ts, state, fill: 4 x [Ly][U][S]
    int32_t* unit = nullptr;  // [Ly][U][kUnitFields]
    int32_t* err = nullptr;
    float* part = nullptr;    // [U][splits][G][D+2], scratch of one step
    double* score = nullptr;  // [U][S] page scores, or [U][S][G] per-head bounds, scratch of one step
    int32_t* fill_att = nullptr;  // [U][S] fills the attention sees (prompt selection), scratch of one step
    int32_t* blist = nullptr;     // [U][Lcap/32] blocks a step visits (prompt selection), likewise
    int32_t* bcnt = nullptr;      // [U][2]
    float* pivl = nullptr;        // [2][U][npr] prompt bound intervals (bf16, fewer units than CUs)
    int npr = 0;                  // prompt region's slots (0: none)
    int nt = 0;                   // K/V blocks streamed with non-temporal loads
    int32_t* seqbuf = nullptr;   // [2][batch] prefill lengths and mask of a ragged prefill
    int32_t* seqhost = nullptr;  // pinned host staging of seqbuf
    hipEvent_t seq_copied = nullptr;  // recorded after the last staging copy
    size_t bytes = 0;
    std::vector<unsigned char> prefilled;
    // Bound on the slots in use, per layer: pages open at the lowest free
    // slot, and no slot is freed before every slot has been used, so a
    // unit that kept k prompt pages and took n decode tokens since uses at
    // most min(S, k + ceil(n / page_size)) slots. keep_max: the most prompt
    // pages any unit of the layer has kept; steps: decode steps of the
    // layer since its first prefill.
    std::vector<int> keep_max;
    std::vector<long long> steps;
    std::vector<unsigned char> descending;  // traversal direction of each layer's next step
    int split_override = 0;
    hipStream_t last_stream = nullptr;
    int prof_mask = 0;
    Timing timing[kKernels];
};

namespace {

// LDS ints the step kernel needs for the prompt selection: a block list of
// the whole pool (list-driven instance), or (in-step selection) the prompt
// pages' bound intervals (two ints each, up to three more to align them to
// 16 bytes), attended fills and blocks, the candidates and their exact
// bounds (two ints each, one more to align them to 8 bytes)
int list_ints(const raas_pool* p) {
    if (p->npr == 0) return 0;
    const int n = p->npr;
    return std::max(p->Lcap / kBlockTokens, 3 + 2 * n + n + n * p->ps / kBlockTokens + n + 1 + 2 * n);
}

LayerView view(const raas_pool* p, int layer) {
    LayerView L;
    const size_t kv = (size_t)layer * p->kv_layer_elems * p->esz;
    const size_t rep = (size_t)layer * p->rep_layer_elems * p->esz;
    const size_t meta = (size_t)layer * p->meta_layer_elems;
    const size_t all_meta = (size_t)p->cfg.n_layers * p->meta_layer_elems;
    L.K = (char*)p->K + kv;
    L.V = (char*)p->V + kv;
    L.kmin = (char*)p->kmin + rep;
    L.kmax = (char*)p->kmax + rep;
    L.lid = p->meta + meta;
    L.ts = p->meta + all_meta + meta;
    L.state = p->meta + 2 * all_meta + meta;
    L.fill = p->meta + 3 * all_meta + meta;
    L.unit = p->unit + (size_t)layer * p->U * kUnitFields;
    L.err = p->err;
    L.score = p->score;
    L.part = p->part;
    L.rev = 0;
    L.nsplit = 1;
    L.bps = p->Lcap / kBlockTokens;
    L.U = p->U;
    L.G = p->G;
    L.D = p->D;
    L.ps = p->ps;
    L.S = p->S;
    L.Lcap = p->Lcap;
    L.bf16 = p->cfg.dtype == RAAS_BF16;
    L.agg = p->cfg.score_aggregation;
    L.rank_pinned = p->cfg.rank_pinned;
    L.hgrp = p->cfg.decision_scope == RAAS_SCOPE_SEQUENCE ? p->cfg.n_kv_heads : 1;
    L.nkv = p->cfg.n_kv_heads;
    L.nblk = p->Lcap / kBlockTokens;
    L.dbase = p->npr;
    L.pcap = p->npr > 0 ? p->npr : p->S - 1;
    L.topk = p->npr > 0 ? p->cfg.prompt_topk : -1;
    L.fill_att = p->npr > 0 ? p->fill_att : L.fill;
    L.blist = p->blist;
    L.bcnt = p->bcnt;
    L.pivl = p->pivl;
    L.pchunk = 0;
    L.lcap_blk = p->Lcap / kBlockTokens;
    L.nt = p->nt;
    L.det = p->cfg.deterministic;
    L.early = 0;
    return L;
}

raas_status validate(const raas_config* c) {
    if (!c) return fail(RAAS_E_INVALID, "cfg is NULL");
    if (c->batch < 1) return fail(RAAS_E_INVALID, "batch must be >= 1 (got %d)", c->batch);
    if (c->n_layers < 1) return fail(RAAS_E_INVALID, "n_layers must be >= 1 (got %d)", c->n_layers);
    if (c->n_kv_heads < 1) return fail(RAAS_E_INVALID, "n_kv_heads must be >= 1 (got %d)", c->n_kv_heads);
    if (c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads != 0)
        return fail(RAAS_E_INVALID, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                    c->n_q_heads, c->n_kv_heads);
    if (c->n_q_heads / c->n_kv_heads > 16)
        return fail(RAAS_E_INVALID, "query group n_q_heads/n_kv_heads = %d exceeds 16",
                    c->n_q_heads / c->n_kv_heads);
    if (c->head_dim != 64 && c->head_dim != 128)
        return fail(RAAS_E_INVALID, "head_dim must be 64 or 128 (got %d)", c->head_dim);
    const int ps = c->page_size;
    if (ps != 8 && ps != 16 && ps != 32 && ps != 64 && ps != 128)
        return fail(RAAS_E_INVALID, "page_size must be 8, 16, 32, 64 or 128 (got %d)", ps);
    if (c->budget_tokens < 1 || c->budget_tokens % ps != 0)
        return fail(RAAS_E_INVALID, "budget_tokens (%d) must be a positive multiple of page_size (%d)",
                    c->budget_tokens, ps);
    if (c->prompt_tokens < 0 || c->prompt_tokens % ps != 0 || c->prompt_tokens % 32 != 0)
        return fail(RAAS_E_INVALID, "prompt_tokens (%d) must be a non-negative multiple of page_size and of 32",
                    c->prompt_tokens);
    if (c->prompt_tokens > 0 && c->prompt_topk < 1)
        return fail(RAAS_E_INVALID, "prompt_topk must be >= 1 with a prompt region (got %d)", c->prompt_topk);
    if (c->prompt_tokens == 0 && c->prompt_topk != 0)
        return fail(RAAS_E_INVALID, "prompt_topk needs a prompt region (prompt_tokens > 0)");
    if (c->deterministic != 0 && c->deterministic != 1)
        return fail(RAAS_E_INVALID, "deterministic must be 0 or 1 (got %d)", c->deterministic);
    if (c->prompt_tokens > 0 && c->rank_pinned)
        return fail(RAAS_E_INVALID, "rank_pinned does not combine with a prompt region");
    const int S = (c->budget_tokens + c->prompt_tokens) / ps;
    if (S < 2 || S > 2048)
        return fail(RAAS_E_INVALID, "(budget_tokens + prompt_tokens) / page_size = %d pages must lie in [2, 2048]",
                    S);
    if (c->dtype != RAAS_F32 && c->dtype != RAAS_BF16)
        return fail(RAAS_E_INVALID, "dtype must be RAAS_F32 or RAAS_BF16 (got %d)", c->dtype);
    if (!(c->r >= 0.0 && c->r <= 1.0)) return fail(RAAS_E_INVALID, "r must lie in [0, 1]");
    if (c->prefill_policy != RAAS_PREFILL_PIN_HEAD && c->prefill_policy != RAAS_PREFILL_ERROR)
        return fail(RAAS_E_INVALID, "unknown prefill_policy %d", c->prefill_policy);
    if (c->score_aggregation != RAAS_SCORE_MAX && c->score_aggregation != RAAS_SCORE_SOFTMAX_SUM)
        return fail(RAAS_E_INVALID, "unknown score_aggregation %d", c->score_aggregation);
    if (c->rank_pinned != 0 && c->rank_pinned != 1)
        return fail(RAAS_E_INVALID, "rank_pinned must be 0 or 1 (got %d)", c->rank_pinned);
    if (c->decision_scope != RAAS_SCOPE_KV_HEAD && c->decision_scope != RAAS_SCOPE_SEQUENCE)
        return fail(RAAS_E_INVALID, "unknown decision_scope %d", c->decision_scope);
    if (c->decision_scope == RAAS_SCOPE_SEQUENCE && c->n_q_heads > 1024)
        return fail(RAAS_E_INVALID, "one decision per sequence covers at most 1024 query heads (got %d)",
                    c->n_q_heads);
    const double units = (double)c->batch * c->n_kv_heads;
    if (units > 1e7) return fail(RAAS_E_INVALID, "batch * n_kv_heads too large");
    return RAAS_OK;
}

raas_status check_layer(const raas_pool* p, int32_t layer) {
    if (!p) return fail(RAAS_E_INVALID, "pool is NULL");
    if (layer < 0 || layer >= p->cfg.n_layers)
        return fail(RAAS_E_INVALID, "layer %d out of range [0, %d)", layer, p->cfg.n_layers);
    return RAAS_OK;
}

// Timing of kernel k's launches (profiling only): a pair of events around
// each launch, in a ring. A HIP failure here never fails the step: events
// that cannot be created switch the kernel's timing off, and a pair whose
// events did not both record is not counted.
void prof_record(raas_pool* p, int k, bool start, hipStream_t s) {
    if (!(p->prof_mask & (1 << k))) return;
    Timing& t = p->timing[k];
    if (t.start.empty()) {
        t.start.assign(kProfRing, nullptr);
        t.stop.assign(kProfRing, nullptr);
        for (size_t i = 0; i < kProfRing; ++i) {
            if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess) {
                (void)hipGetLastError();
                p->prof_mask &= ~(1 << k);
                return;  // (raas_destroy releases the events created so far)
            }
        }
    }
    const size_t slot = (t.head + t.count) % kProfRing;
    if (start) {
        if (t.count == kProfRing) {  // recycle the oldest pair
            float ms = 0.f;
            if (hipEventSynchronize(t.stop[t.head]) == hipSuccess &&
                hipEventElapsedTime(&ms, t.start[t.head], t.stop[t.head]) == hipSuccess) {
                t.folded_ms += ms;
                t.folded_n += 1;
            }
            t.head = (t.head + 1) % kProfRing;
            t.count -= 1;
        }
        t.started = hipEventRecord(t.start[(t.head + t.count) % kProfRing], s) == hipSuccess;
    } else {
        if (t.started && hipEventRecord(t.stop[slot], s) == hipSuccess) t.count += 1;
        t.started = false;
    }
}

// The step's scratch in the fixed device array of raas_decode_step_static:
// the split partials, the page scores, and the prompt selection's attended
// fills, block lists and counts, each 256-byte aligned.
__device__ __align__(256) unsigned char scratch[RAAS_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // scratch's device address, per device

// Address of this device's copy of `scratch` (looked up once per device,
// with the device current; the array's name is no device address in host
// code).
raas_status static_scratch(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(RAAS_E_INVALID, "device %d beyond the static scratch table", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return RAAS_OK;
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// One decode step of one layer (raas_decode_step_masked); with
// fixed_scratch the per-step scratch comes from `scratch` instead of the
// pool's buffers, and nothing is allocated or profiled.
raas_status decode_step(raas_pool* p, int32_t layer, const StepIO& io, hipStream_t s, bool fixed_scratch) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    if (!io.q || !io.k_new || !io.v_new || !io.out)
        return fail(RAAS_E_INVALID, "q, k_new, v_new and out must be non-NULL");
    if (!p->prefilled[layer]) return fail(RAAS_E_STATE, "layer %d has not been prefilled", layer);
    LayerView L = view(p, layer);
    // visit only the blocks that can hold resident rows (see keep_max)
    const long long pages_opened = (p->steps[layer] + 1 + p->ps - 1) / p->ps;
    const long long used = std::min<long long>(p->S, p->keep_max[layer] + pages_opened);
    L.nblk = (int)std::min<long long>(p->Lcap / kBlockTokens, (used * p->ps + kBlockTokens - 1) / kBlockTokens);
    // blocks the step attends: with a prompt region only the chosen prompt
    // pages' blocks (at most topk pages, each on ceil(page_size / 32) blocks)
    int work_blocks = L.nblk;
    if (p->npr > 0) {
        const int nbp = p->npr * p->ps / kBlockTokens;
        const int per_page = std::max(1, p->ps / kBlockTokens);
        work_blocks = L.nblk - nbp + std::min(nbp, p->cfg.prompt_topk * per_page);
    }
    const StepPlan pl = plan_step(p->U, p->G, p->D, p->S, L.nblk * kBlockTokens, p->ps, work_blocks,
                                  p->cfg.dtype == RAAS_BF16, p->cfg.score_aggregation,
                                  p->cfg.decision_scope == RAAS_SCOPE_SEQUENCE, list_ints(p), p->split_override, p->npr);
    L.nsplit = pl.nsplit;
    L.bps = pl.bps;
    // the first score pass issued with the first blocks: the score barrier and
    // the retention come a block sooner, which pays where a workgroup of 8
    // wavefronts streams at least 8 blocks each (batch 32 at L 2048: 40.79 ->
    // 40.38 us, the Qwen stack and L 8192 level) and not below (batch 1 at
    // L 1024 +0.14 us; batch 128 at L 512, 2 wavefronts, +0.23 us)
    L.early = pl.waves == 8 && L.nblk >= 8 * pl.waves ? 1 : 0;
    const bool select_kernel = p->npr > 0 && !pl.select_in_step;
    if (fixed_scratch) {
        const size_t U = (size_t)p->U, S = (size_t)p->S;
        const size_t part = pl.fused ? 0 : align256(U * pl.nsplit * p->G * (p->D + 2) * sizeof(float));
        const size_t score =
            pl.fused ? 0 : align256(U * S * (p->cfg.score_aggregation == RAAS_SCORE_SOFTMAX_SUM ? p->G : 1) * 8);
        const size_t fatt = select_kernel ? align256(U * S * 4) : 0;
        const size_t blist = select_kernel ? align256(U * (p->Lcap / kBlockTokens) * 4) : 0;
        const size_t bcnt = select_kernel ? align256(U * 2 * 4) : 0;
        const size_t need = part + score + fatt + blist + bcnt;
        if (need > RAAS_STATIC_SCRATCH_BYTES)
            return fail(RAAS_E_INVALID, "this step needs %zu bytes of scratch; the static array holds %u", need,
                        (unsigned)RAAS_STATIC_SCRATCH_BYTES);
        if (need > 0) {
            void* base = nullptr;
            st = static_scratch(&base);
            if (st != RAAS_OK) return st;
            char* c = (char*)base;
            L.part = part ? (float*)c : nullptr;
            L.score = score ? (double*)(c + part) : nullptr;
            if (select_kernel) {
                L.fill_att = (int32_t*)(c + part + score);
                L.blist = (int32_t*)(c + part + score + fatt);
                L.bcnt = (int32_t*)(c + part + score + fatt + blist);
            }
        }
    }
    // Successive steps of a layer read its pool in opposite directions, so a
    // step starts with the blocks the previous one read last, the likeliest
    // to be still in the GPU's memory-side cache.
    L.rev = p->descending[layer];
    const bool prof = !fixed_scratch;

    if (select_kernel) {  // Quest on the prompt: which prompt pages this step attends to
        // Fewer units than CUs and a long prompt region (bf16): the prompt
        // pages' bound intervals first, by a kernel of single-wavefront
        // workgroups of 32 or more pages each, up to about eight per CU (the
        // selection kernel would draw them on one CU per unit); not with the
        // static scratch, which holds no intervals.
        if (!fixed_scratch && p->cfg.dtype == RAAS_BF16 && p->U < 256 && p->npr > 256) {
            const int per = (p->npr * p->U + 2047) / 2048;
            L.pchunk = std::max(32, (per + 15) / 16 * 16);
        }
        if (prof) prof_record(p, 2, true, s);
        hipError_t e = launch_prompt_select(L, io, s);
        if (prof) prof_record(p, 2, false, s);
        if (e != hipSuccess) return hip_fail(e, "prompt selection launch");
    }
    if (prof) prof_record(p, 0, true, s);
    hipError_t e = launch_step(L, io, pl, p->cfg.r, s);
    if (prof) prof_record(p, 0, false, s);
    if (e != hipSuccess) return hip_fail(e, "step launch");
    if (!pl.fused) {
        if (prof) prof_record(p, 1, true, s);
        e = launch_epilogue(L, io, p->cfg.r, s);
        if (prof) prof_record(p, 1, false, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue launch");
    }
    p->descending[layer] ^= 1;
    p->steps[layer] += 1;
    p->last_stream = s;
    return RAAS_OK;
}

}  // namespace

extern "C" {

const char* raas_last_error(void) { return g_last_error.c_str(); }

int32_t raas_abi_version(void) { return RAAS_ABI_VERSION; }

size_t raas_pool_bytes(const raas_pool* p) { return p ? p->bytes : 0; }

raas_status raas_create_pool(const raas_config* cfg, void* stream, raas_pool** out) {
    if (!out) return fail(RAAS_E_INVALID, "out is NULL");
    raas_status st = validate(cfg);
    if (st != RAAS_OK) return st;
    raas_pool* p = new (std::nothrow) raas_pool();
    if (!p) return fail(RAAS_E_OOM, "host allocation failed");
    p->cfg = *cfg;
    p->U = cfg->batch * cfg->n_kv_heads;
    p->G = cfg->n_q_heads / cfg->n_kv_heads;
    p->D = cfg->head_dim;
    p->ps = cfg->page_size;
    p->S = (cfg->budget_tokens + cfg->prompt_tokens) / cfg->page_size;
    p->npr = cfg->prompt_tokens / cfg->page_size;
    p->Lcap = (p->S * p->ps + kBlockTokens - 1) / kBlockTokens * kBlockTokens;
    p->esz = cfg->dtype == RAAS_BF16 ? 2 : 4;
    p->kv_layer_elems = (size_t)p->U * p->Lcap * p->D;
    p->rep_layer_elems = (size_t)p->U * p->S * p->D;
    p->meta_layer_elems = (size_t)p->U * p->S;
    p->prefilled.assign((size_t)cfg->n_layers, 0);
    p->keep_max.assign((size_t)cfg->n_layers, 0);
    p->steps.assign((size_t)cfg->n_layers, 0);
    p->descending.assign((size_t)cfg->n_layers, 0);
    // A step reads a layer's whole pool; the same layer comes round again
    // after every layer's pool has been read. When all of them exceed twice
    // the memory-side cache (256 MB), nothing of a step's reads is left there
    // for the next: the blocks are then read with non-temporal loads, which
    // stream faster. Smaller pools keep ordinary loads and the cache's reuse.
    p->nt = 2.0 * (double)cfg->n_layers * p->U * p->Lcap * p->D * p->esz > 2.0 * 256e6 ? 1 : 0;
    const size_t Ly = (size_t)cfg->n_layers;
    const int nblk = p->Lcap / kBlockTokens;
    const int max_split = nblk < kMaxSplits ? nblk : kMaxSplits;
    struct Req {
        void** ptr;
        size_t bytes;
    } reqs[] = {
        {&p->K, Ly * p->kv_layer_elems * p->esz},
        {&p->V, Ly * p->kv_layer_elems * p->esz},
        {&p->kmin, Ly * p->rep_layer_elems * p->esz},
        {&p->kmax, Ly * p->rep_layer_elems * p->esz},
        {(void**)&p->meta, 4 * Ly * p->meta_layer_elems * sizeof(int32_t)},
        {(void**)&p->unit, Ly * p->U * kUnitFields * sizeof(int32_t)},
        {(void**)&p->err, 256},
        {(void**)&p->part, (size_t)p->U * max_split * p->G * (p->D + 2) * sizeof(float)},
        {(void**)&p->score,
         (size_t)p->U * p->S * (cfg->score_aggregation == RAAS_SCORE_SOFTMAX_SUM ? p->G : 1) * sizeof(double)},
        {(void**)&p->seqbuf, 2 * (size_t)cfg->batch * sizeof(int32_t)},
        {(void**)&p->fill_att, p->npr > 0 ? (size_t)p->U * p->S * sizeof(int32_t) : 4},
        {(void**)&p->blist, p->npr > 0 ? (size_t)p->U * (p->Lcap / kBlockTokens) * sizeof(int32_t) : 4},
        {(void**)&p->bcnt, p->npr > 0 ? (size_t)p->U * 2 * sizeof(int32_t) : 4},
        {(void**)&p->pivl, p->npr > 0 ? 2 * (size_t)p->U * p->npr * sizeof(float) : 4},
    };
    hipStream_t s = (hipStream_t)stream;
    hipError_t ea = allow_large_lds();
    if (ea != hipSuccess) {
        raas_destroy(p);
        return hip_fail(ea, "hipFuncSetAttribute");
    }
    for (auto& r : reqs) {
        hipError_t e = hipMalloc(r.ptr, r.bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            raas_destroy(p);
            return fail(e == hipErrorOutOfMemory ? RAAS_E_OOM : RAAS_E_HIP, "hipMalloc(%zu bytes): %s",
                        r.bytes, hipGetErrorString(e));
        }
        p->bytes += r.bytes;
        e = hipMemsetAsync(*r.ptr, 0, r.bytes, s);
        if (e != hipSuccess) {
            raas_destroy(p);
            return hip_fail(e, "hipMemsetAsync");
        }
    }
    hipError_t eh = hipHostMalloc((void**)&p->seqhost, 2 * (size_t)cfg->batch * sizeof(int32_t));
    if (eh != hipSuccess) {
        p->seqhost = nullptr;
        raas_destroy(p);
        return fail(RAAS_E_OOM, "hipHostMalloc: %s", hipGetErrorString(eh));
    }
    // every slot starts free: lid = ts = -1, state = free (0), fill = 0
    hipError_t e = hipMemsetAsync(p->meta, 0xFF, 2 * Ly * p->meta_layer_elems * sizeof(int32_t), s);
    if (e != hipSuccess) {
        raas_destroy(p);
        return hip_fail(e, "hipMemsetAsync");
    }
    p->last_stream = s;
    *out = p;
    return RAAS_OK;
}

void raas_destroy(raas_pool* p) {
    if (!p) return;
    // the pool's work has run before its memory goes; a failure here (a
    // device already lost) leaves nothing else to undo, so it is not reported
    if (p->K || p->meta) (void)hipStreamSynchronize(p->last_stream);
    for (auto& t : p->timing) {
        for (auto ev : t.start)
            if (ev) (void)hipEventDestroy(ev);
        for (auto ev : t.stop)
            if (ev) (void)hipEventDestroy(ev);
    }
    void* ptrs[] = {p->K,     p->V,     p->kmin,  p->kmax,     p->meta,  p->unit, p->err,
                    p->part,  p->score, p->seqbuf, p->fill_att, p->blist, p->bcnt, p->pivl};
    for (void* q : ptrs)
        if (q) (void)hipFree(q);
    if (p->seqhost) (void)hipHostFree(p->seqhost);
    if (p->seq_copied) (void)hipEventDestroy(p->seq_copied);
    delete p;
}

raas_status raas_prefill(raas_pool* p, int32_t layer, const void* k, const void* v,
                         int32_t prefill_len, void* stream) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    if (prefill_len < 0) return fail(RAAS_E_INVALID, "prefill_len must be >= 0 (got %d)", prefill_len);
    if (prefill_len > 0 && (!k || !v)) return fail(RAAS_E_INVALID, "k or v is NULL");
    if (p->prefilled[layer]) return fail(RAAS_E_STATE, "layer %d was already prefilled", layer);
    const int pages = (prefill_len + p->ps - 1) / p->ps;
    const int pcap = p->npr > 0 ? p->npr : p->S - 1;  // S-1: one slot stays for decode pages
    int keep = pages;
    if (keep > pcap) {
        if (p->cfg.prefill_policy == RAAS_PREFILL_ERROR)
            return fail(RAAS_E_BUDGET, "prefill needs %d pages but %d are available to it", pages, pcap);
        keep = pcap;
    }
    hipStream_t s = (hipStream_t)stream;
    const PrefillIn in{nullptr, nullptr, prefill_len, prefill_len};
    hipError_t e = launch_prefill(view(p, layer), k, v, in, std::min(prefill_len, keep * p->ps), s);
    if (e != hipSuccess) return hip_fail(e, "prefill launch");
    p->prefilled[layer] = 1;
    p->keep_max[layer] = std::max(keep, p->npr);  // decode pages start after the prompt region
    p->steps[layer] = 0;
    p->last_stream = s;
    return RAAS_OK;
}

raas_status raas_prefill_ragged(raas_pool* p, int32_t layer, const void* k, const void* v,
                                const int32_t* prefill_lens, const int32_t* seq_mask, int32_t max_len,
                                void* stream) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    if (!prefill_lens) return fail(RAAS_E_INVALID, "prefill_lens is NULL");
    if (max_len < 0) return fail(RAAS_E_INVALID, "max_len must be >= 0 (got %d)", max_len);
    const int B = p->cfg.batch;
    int max_tok = 0, selected = 0, keep_max = 0;
    for (int b = 0; b < B; ++b) {
        if (seq_mask && !seq_mask[b]) continue;
        ++selected;
        const int P = prefill_lens[b];
        if (P < 0 || P > max_len)
            return fail(RAAS_E_INVALID, "prefill_lens[%d] = %d outside [0, max_len = %d]", b, P, max_len);
        const int pages = (P + p->ps - 1) / p->ps;
        const int pcap = p->npr > 0 ? p->npr : p->S - 1;
        if (pages > pcap && p->cfg.prefill_policy == RAAS_PREFILL_ERROR)
            return fail(RAAS_E_BUDGET, "sequence %d: prefill needs %d pages but %d are available to it", b, pages,
                        pcap);
        max_tok = std::max(max_tok, std::min(P, std::min(pages, pcap) * p->ps));
        keep_max = std::max(keep_max, std::max(std::min(pages, pcap), p->npr));
    }
    if (!p->prefilled[layer] && selected != B)
        return fail(RAAS_E_STATE, "the first prefill of layer %d must cover every sequence", layer);
    if (max_tok > 0 && (!k || !v)) return fail(RAAS_E_INVALID, "k or v is NULL");
    hipStream_t s = (hipStream_t)stream;
    // lengths and mask go to the device through the pool's pinned staging
    // buffer, once the previous ragged prefill's copy out of it has run
    hipError_t e = hipSuccess;
    if (!p->seq_copied) {
        e = hipEventCreateWithFlags(&p->seq_copied, hipEventDisableTiming);
        if (e != hipSuccess) {
            p->seq_copied = nullptr;
            return hip_fail(e, "hipEventCreateWithFlags");
        }
    } else {
        e = hipEventSynchronize(p->seq_copied);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    }
    for (int b = 0; b < B; ++b) {
        p->seqhost[b] = prefill_lens[b];
        p->seqhost[(size_t)B + b] = (seq_mask && !seq_mask[b]) ? 0 : 1;
    }
    e = hipMemcpyAsync(p->seqbuf, p->seqhost, 2 * (size_t)B * sizeof(int32_t), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
    e = hipEventRecord(p->seq_copied, s);
    if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
    const PrefillIn in{p->seqbuf, p->seqbuf + B, 0, max_len};
    e = launch_prefill(view(p, layer), k, v, in, max_tok, s);
    if (e != hipSuccess) return hip_fail(e, "prefill launch");
    if (!p->prefilled[layer]) {
        p->keep_max[layer] = keep_max;
        p->steps[layer] = 0;
    } else {
        p->keep_max[layer] = std::max(p->keep_max[layer], keep_max);
    }
    p->prefilled[layer] = 1;
    p->last_stream = s;
    return RAAS_OK;
}

raas_status raas_decode_step(raas_pool* p, int32_t layer, const void* q, const void* k_new,
                             const void* v_new, void* out, int32_t* page_table_out,
                             int32_t* timestamps_out, int32_t* evicted_out, void* stream) {
    return raas_decode_step_masked(p, layer, q, k_new, v_new, out, page_table_out, timestamps_out, evicted_out,
                                   nullptr, stream);
}

raas_status raas_decode_step_masked(raas_pool* p, int32_t layer, const void* q, const void* k_new,
                                    const void* v_new, void* out, int32_t* page_table_out,
                                    int32_t* timestamps_out, int32_t* evicted_out, const int32_t* active,
                                    void* stream) {
    const StepIO io{q, k_new, v_new, out, page_table_out, timestamps_out, evicted_out, active};
    return decode_step(p, layer, io, (hipStream_t)stream, false);
}

raas_status raas_decode_step_static(raas_pool* p, int32_t layer, const void* q, const void* k_new,
                                    const void* v_new, void* out, int32_t* page_table_out,
                                    int32_t* timestamps_out, int32_t* evicted_out, void* stream) {
    const StepIO io{q, k_new, v_new, out, page_table_out, timestamps_out, evicted_out, nullptr};
    return decode_step(p, layer, io, (hipStream_t)stream, true);
}

raas_status raas_export_state(raas_pool* p, int32_t layer, int32_t* host_buf, size_t n_ints,
                              void* stream) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    const size_t need = (size_t)p->U * (4 * (size_t)p->S + 4);
    if (!host_buf || n_ints != need)
        return fail(RAAS_E_INVALID, "host_buf must hold %zu int32 (got %zu)", need, n_ints);
    const LayerView L = view(p, layer);
    hipStream_t s = (hipStream_t)stream;
    const size_t us = (size_t)p->U * p->S;
    int32_t* src[4] = {L.lid, L.ts, L.state, L.fill};
    for (int i = 0; i < 4; ++i) {
        hipError_t e = hipMemcpyAsync(host_buf + i * us, src[i], us * sizeof(int32_t), hipMemcpyDeviceToHost, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
    }
    std::vector<int32_t> unit((size_t)p->U * kUnitFields);
    hipError_t e = hipMemcpyAsync(unit.data(), L.unit, unit.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
    int32_t errflag = 0;
    e = hipMemcpyAsync(&errflag, p->err, sizeof(int32_t), hipMemcpyDeviceToHost, s);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    if (errflag) return fail(RAAS_E_HIP, "device reported an internal inconsistency (flag %d)", errflag);
    for (int u = 0; u < p->U; ++u)
        for (int f = 0; f < 4; ++f) host_buf[4 * us + 4 * (size_t)u + f] = unit[(size_t)u * kUnitFields + f];
    return RAAS_OK;
}

namespace {

// Checkpoint layout: a header, then the layer's device sections in order
// (K, V, kmin, kmax, lid, ts, state, fill, unit records), each 256-byte
// aligned in the buffer.
constexpr uint64_t kCkptMagic = 0x54504b4353414152ull;  // "RAASCKPT"
struct CkptHeader {
    uint64_t magic;
    int64_t abi, bytes;
    int64_t cfg[16];  // the configuration, field by field
    int64_t prefilled, keep_max, steps, descending;
};

void ckpt_config(const raas_config& c, int64_t* out) {
    const int64_t f[16] = {c.batch, c.n_layers, c.n_q_heads, c.n_kv_heads, c.head_dim, c.page_size,
                           c.budget_tokens, c.dtype, (int64_t)llround(c.r * 1e12), c.prefill_policy,
                           c.score_aggregation, c.rank_pinned, c.decision_scope, c.prompt_tokens, c.prompt_topk,
                           c.deterministic};
    memcpy(out, f, sizeof f);
}

struct CkptSection {
    void* dev;
    size_t bytes;
};

// The device sections of one layer, in checkpoint order; returns their count.
int ckpt_sections(const raas_pool* p, int layer, CkptSection* out) {
    const LayerView L = view(p, layer);
    const size_t kv = p->kv_layer_elems * p->esz, rep = p->rep_layer_elems * p->esz;
    const size_t meta = p->meta_layer_elems * sizeof(int32_t);
    const CkptSection sec[9] = {{L.K, kv},        {L.V, kv},          {L.kmin, rep},
                                {L.kmax, rep},    {L.lid, meta},      {L.ts, meta},
                                {L.state, meta},  {L.fill, meta},     {L.unit, (size_t)p->U * kUnitFields * 4}};
    memcpy(out, sec, sizeof sec);
    return 9;
}

size_t ckpt_bytes(const raas_pool* p) {
    CkptSection sec[9];
    const int n = ckpt_sections(p, 0, sec);
    size_t b = align256(sizeof(CkptHeader));
    for (int i = 0; i < n; ++i) b += align256(sec[i].bytes);
    return b;
}

}  // namespace

size_t raas_layer_checkpoint_bytes(const raas_pool* p) { return p ? ckpt_bytes(p) : 0; }

raas_status raas_save_layer(raas_pool* p, int32_t layer, void* host_buf, size_t bytes, void* stream) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    if (!host_buf || bytes != ckpt_bytes(p))
        return fail(RAAS_E_INVALID, "host_buf must hold %zu bytes (got %zu)", ckpt_bytes(p), bytes);
    CkptHeader h{};
    h.magic = kCkptMagic;
    h.abi = RAAS_ABI_VERSION;
    h.bytes = (int64_t)bytes;
    ckpt_config(p->cfg, h.cfg);
    h.prefilled = p->prefilled[layer];
    h.keep_max = p->keep_max[layer];
    h.steps = p->steps[layer];
    h.descending = p->descending[layer];
    memcpy(host_buf, &h, sizeof h);
    hipStream_t s = (hipStream_t)stream;
    CkptSection sec[9];
    const int n = ckpt_sections(p, layer, sec);
    size_t off = align256(sizeof h);
    for (int i = 0; i < n; ++i) {
        hipError_t e = hipMemcpyAsync((char*)host_buf + off, sec[i].dev, sec[i].bytes, hipMemcpyDeviceToHost, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
        off += align256(sec[i].bytes);
    }
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    return RAAS_OK;
}

raas_status raas_load_layer(raas_pool* p, int32_t layer, const void* host_buf, size_t bytes, void* stream) {
    raas_status st = check_layer(p, layer);
    if (st != RAAS_OK) return st;
    if (!host_buf || bytes != ckpt_bytes(p))
        return fail(RAAS_E_INVALID, "host_buf must hold %zu bytes (got %zu)", ckpt_bytes(p), bytes);
    CkptHeader h;
    memcpy(&h, host_buf, sizeof h);
    int64_t cfg[16];
    ckpt_config(p->cfg, cfg);
    if (h.magic != kCkptMagic) return fail(RAAS_E_INVALID, "not a layer checkpoint");
    if (h.abi != RAAS_ABI_VERSION || h.bytes != (int64_t)bytes)
        return fail(RAAS_E_INVALID, "checkpoint of ABI %lld, %lld bytes", (long long)h.abi, (long long)h.bytes);
    if (memcmp(h.cfg, cfg, sizeof cfg) != 0)
        return fail(RAAS_E_INVALID, "checkpoint of a pool with another configuration");
    if ((h.prefilled != 0 && h.prefilled != 1) || h.keep_max < 0 || h.keep_max > p->S || h.steps < 0 ||
        (h.descending != 0 && h.descending != 1))
        return fail(RAAS_E_INVALID, "corrupt checkpoint header");
    hipStream_t s = (hipStream_t)stream;
    CkptSection sec[9];
    const int n = ckpt_sections(p, layer, sec);
    size_t off = align256(sizeof h);
    for (int i = 0; i < n; ++i) {
        hipError_t e =
            hipMemcpyAsync(sec[i].dev, (const char*)host_buf + off, sec[i].bytes, hipMemcpyHostToDevice, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
        off += align256(sec[i].bytes);
    }
    p->prefilled[layer] = (unsigned char)h.prefilled;
    p->keep_max[layer] = (int)h.keep_max;
    p->steps[layer] = h.steps;
    p->descending[layer] = (unsigned char)h.descending;
    p->last_stream = s;
    return RAAS_OK;
}

raas_status raas_set_attention_splits(raas_pool* p, int32_t splits) {
    if (!p) return fail(RAAS_E_INVALID, "pool is NULL");
    if (splits < 0 || splits > kMaxSplits) return fail(RAAS_E_INVALID, "splits must lie in [0, %d]", kMaxSplits);
    p->split_override = splits;
    return RAAS_OK;
}

raas_status raas_profile(raas_pool* p, int32_t mask) {
    if (!p) return fail(RAAS_E_INVALID, "pool is NULL");
    if (mask < 0 || mask >= (1 << kKernels)) return fail(RAAS_E_INVALID, "bad kernel mask %d", mask);
    p->prof_mask = mask;
    return RAAS_OK;
}

raas_status raas_profile_read(raas_pool* p, int32_t kernel, double* total_ms, int64_t* launches) {
    if (!p) return fail(RAAS_E_INVALID, "pool is NULL");
    if (kernel < 0 || kernel >= kKernels || !total_ms || !launches)
        return fail(RAAS_E_INVALID, "bad kernel index or NULL output");
    Timing& t = p->timing[kernel];
    double ms_sum = t.folded_ms;
    int64_t n = t.folded_n;
    for (size_t i = 0; i < t.count; ++i) {
        const size_t j = (t.head + i) % kProfRing;
        hipError_t e = hipEventSynchronize(t.stop[j]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, t.start[j], t.stop[j]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        ms_sum += ms;
        n += 1;
    }
    t.head = 0;
    t.count = 0;
    t.folded_ms = 0.0;
    t.folded_n = 0;
    *total_ms = ms_sum;
    *launches = n;
    return RAAS_OK;
}

}  // extern "C"
