// Streaming probe (measurement only, not part of the decode path): reads a
// buffer laid out as the step kernel's K/V pool -- per unit a run of 32-token
// blocks of 16 KB (d 128) or 8 KB (d 64), K and V in separate arrays -- with
// the step kernel's access structure and no arithmetic, so that its rate
// bounds what the step kernel can reach on the same data. A workgroup of NW
// wavefronts reads one unit: each wavefront takes block w, then claims further
// blocks (from a counter in LDS, or a fixed interleave), with the next block's
// loads issued before the current one is consumed. MODE 0 holds that next
// block in registers (as the step kernel does); MODE 1 stages it in LDS with
// direct global-to-LDS loads instead, two blocks per wavefront in flight. The
// loaded words are folded into one word per wavefront so that no load is
// dropped. Launches read the layers' pools in turn, alternating the traversal
// direction per layer if asked.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "raas_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// s_waitcnt operand: vmcnt(n), expcnt and lgkmcnt left at their maxima
constexpr int vmcnt(int n) { return (n & 0xF) | ((n >> 4) << 14) | 0x70 | 0xF00; }

template <bool NT>
__device__ __forceinline__ u32x4 ldg(const uint16_t* p) {
    if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    else return *reinterpret_cast<const u32x4*>(p);
}

// one block's loads of one lane: 2*D/32 K vectors and D/16 V vectors of 16 bytes
template <int D>
struct Blk {
    u32x4 k[D / 16], v[D / 16];
};

template <int D, int NW, bool NT, int MODE>
__global__ __launch_bounds__(NW * 64) void k_probe(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                                   int lcap_blk, int nblk, int rev, int dyn, int kvi, unsigned* sink) {
    constexpr int BLK = 32 * D;  // elements of K (or V) per block
    constexpr int NV = D / 16;   // 16-byte vectors per lane per array
    __shared__ int s_next;
    extern __shared__ __align__(16) unsigned char stage[];  // MODE 1: [NW][2][2 * NV * 64] 16-byte vectors
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // kvi: block b's K at K + (u * lcap_blk + b) * 2 * BLK, its V right after (the buffer K spans both)
    const size_t bstride = kvi ? 2 * BLK : BLK;
    const uint16_t* Ku = K + (size_t)blockIdx.x * lcap_blk * bstride;
    const uint16_t* Vu = kvi ? Ku + BLK : V + (size_t)blockIdx.x * lcap_blk * BLK;
    if (threadIdx.x == 0) s_next = 2 * NW;
    __syncthreads();
    auto blk_of = [&](int i) { return rev ? nblk - 1 - i : i; };
    int it = 0;
    auto claim = [&]() {
        int c;
        if (dyn) {
            c = 0;
            if (lane == 0) c = it == 0 ? w + NW : atomicAdd(&s_next, 1);
            c = __builtin_amdgcn_readfirstlane(c);
        } else {
            c = w + (it + 1) * NW;
        }
        ++it;
        return c;
    };
    unsigned acc = 0;
    if constexpr (MODE == 0) {
        Blk<D> nx;
        auto load = [&](int b) {
            const uint16_t* kb = Ku + (size_t)b * bstride + lane * 8;
            const uint16_t* vb = Vu + (size_t)b * bstride + lane * 8;
#pragma unroll
            for (int i = 0; i < NV; ++i) nx.k[i] = ldg<NT>(kb + i * 512);
#pragma unroll
            for (int i = 0; i < NV; ++i) nx.v[i] = ldg<NT>(vb + i * 512);
        };
        int i = w;
        if (i < nblk) load(blk_of(i));
        while (i < nblk) {
            Blk<D> cur = nx;
            const int n = claim();
            if (n < nblk) load(blk_of(n));
#pragma unroll
            for (int j = 0; j < NV; ++j) acc ^= cur.k[j].x ^ cur.k[j].w ^ cur.v[j].y ^ cur.v[j].z;
            i = n;
        }
    } else {
        // two LDS slots per wavefront; slot s of wavefront w at stage + ((w * 2 + s) * 2 * NV * 64) * 16
        auto slot = [&](int s) {
            return reinterpret_cast<u32x4*>(stage) + (size_t)(w * 2 + s) * 2 * NV * 64;
        };
        auto issue = [&](int b, int s) {  // block b's 2 * NV wave-wide 1 KB rows into slot s
            const uint16_t* kb = Ku + (size_t)b * bstride + lane * 8;
            const uint16_t* vb = Vu + (size_t)b * bstride + lane * 8;
            u32x4* dst = slot(s);
#pragma unroll
            for (int j = 0; j < NV; ++j)
                __builtin_amdgcn_global_load_lds(kb + j * 512, (__attribute__((address_space(3))) void*)(dst + j * 64),
                                                 16, 0, NT ? 2 : 0);
#pragma unroll
            for (int j = 0; j < NV; ++j)
                __builtin_amdgcn_global_load_lds(vb + j * 512,
                                                 (__attribute__((address_space(3))) void*)(dst + (NV + j) * 64), 16, 0,
                                                 NT ? 2 : 0);
        };
        int i0 = w, i1 = nblk;
        if (i0 < nblk) issue(blk_of(i0), 0);
        if (i0 < nblk) {
            i1 = claim();
            if (i1 < nblk) issue(blk_of(i1), 1);
        }
        int s = 0;
        while (i0 < nblk) {
            // the older block's loads are complete once at most the newer block's are outstanding
            if (i1 < nblk) __builtin_amdgcn_s_waitcnt(vmcnt(2 * NV));
            else __builtin_amdgcn_s_waitcnt(vmcnt(0));
            const u32x4* src = slot(s);
            Blk<D> cur;
#pragma unroll
            for (int j = 0; j < NV; ++j) cur.k[j] = src[j * 64 + lane];
#pragma unroll
            for (int j = 0; j < NV; ++j) cur.v[j] = src[(NV + j) * 64 + lane];
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): the slot has been read
            const int n = i1 < nblk ? claim() : nblk;
            if (n < nblk) issue(blk_of(n), s);
#pragma unroll
            for (int j = 0; j < NV; ++j) acc ^= cur.k[j].x ^ cur.k[j].w ^ cur.v[j].y ^ cur.v[j].z;
            i0 = i1;
            i1 = n;
            s ^= 1;
        }
    }
    sink[blockIdx.x * NW + w] = acc;
}

template <int D, int NW, bool NT, int MODE>
void launch(const raas_probe_config& c, const uint16_t* K, const uint16_t* V, int lcap_blk, int nblk, int rev,
            unsigned* sink, hipStream_t s) {
    const size_t lds = MODE == 1 ? (size_t)NW * 2 * 2 * (D / 16) * 64 * 16 : 0;
    hipLaunchKernelGGL((k_probe<D, NW, NT, MODE>), dim3(c.units), dim3(NW * 64), lds, s, K, V, lcap_blk, nblk, rev,
                       c.dynamic, c.kv_interleaved, sink);
}

template <int D, int NW>
bool launch_nw(const raas_probe_config& c, const uint16_t* K, const uint16_t* V, int lcap_blk, int nblk, int rev,
               unsigned* sink, hipStream_t s) {
    if (c.mode == 0 && !c.nontemporal) launch<D, NW, false, 0>(c, K, V, lcap_blk, nblk, rev, sink, s);
    else if (c.mode == 0) launch<D, NW, true, 0>(c, K, V, lcap_blk, nblk, rev, sink, s);
    else if (!c.nontemporal) launch<D, NW, false, 1>(c, K, V, lcap_blk, nblk, rev, sink, s);
    else launch<D, NW, true, 1>(c, K, V, lcap_blk, nblk, rev, sink, s);
    return true;
}

template <int NW>
bool set_lds() {
    const int b = NW * 2 * 2 * 8 * 64 * 16;
    return hipFuncSetAttribute((const void*)k_probe<128, NW, false, 1>, hipFuncAttributeMaxDynamicSharedMemorySize, b) ==
               hipSuccess &&
           hipFuncSetAttribute((const void*)k_probe<128, NW, true, 1>, hipFuncAttributeMaxDynamicSharedMemorySize, b) ==
               hipSuccess;
}

}  // namespace

extern "C" int raas_probe_stream(const raas_probe_config* c, double* us_per_launch, double* bytes_per_launch) {
    if (!c || !us_per_launch || !bytes_per_launch) return -1;
    if (c->units < 1 || c->tokens < 32 || c->tokens % 32 || c->layers < 1 || c->launches < 1) return -1;
    if (c->head_dim != 64 && c->head_dim != 128) return -1;
    if (c->waves != 2 && c->waves != 4 && c->waves != 8) return -1;
    if (c->mode != 0 && c->mode != 1) return -1;
    if (c->kv_interleaved != 0 && c->kv_interleaved != 1) return -1;
    if (c->mode == 1 && (c->head_dim != 128 || c->waves > 4)) return -1;  // two 16 KB slots per wavefront
    const int lcap_blk = c->tokens / 32, nblk = lcap_blk;
    const size_t per_layer = (size_t)c->units * c->tokens * c->head_dim;  // elements of K (or V)
    uint16_t *K = nullptr, *V = nullptr;
    unsigned* sink = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    int rc = -2;
    const int kvi = c->kv_interleaved ? 1 : 0;  // K holds both halves; V is unused
    if (hipMalloc(&K, per_layer * c->layers * 2 * (1 + kvi)) != hipSuccess) K = nullptr;
    if (hipMalloc(&V, kvi ? 256 : per_layer * c->layers * 2) != hipSuccess) V = nullptr;
    if (hipMalloc(&sink, (size_t)c->units * 8 * sizeof(unsigned)) != hipSuccess) sink = nullptr;
    if (K && V && sink && hipMemset(K, 0x3C, per_layer * c->layers * 2 * (1 + kvi)) == hipSuccess &&
        hipMemset(V, 0x3C, kvi ? 256 : per_layer * c->layers * 2) == hipSuccess && hipEventCreate(&e0) == hipSuccess &&
        hipEventCreate(&e1) == hipSuccess && set_lds<2>() && set_lds<4>()) {
        auto run = [&](int i) {
            const int layer = i % c->layers;
            const int rev = c->alternate ? (i / c->layers) & 1 : 0;
            const uint16_t* Kl = K + per_layer * layer * (1 + kvi);
            const uint16_t* Vl = kvi ? V : V + per_layer * layer;
            hipStream_t s = nullptr;
            if (c->head_dim == 128) {
                if (c->waves == 8) launch_nw<128, 8>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
                else if (c->waves == 4) launch_nw<128, 4>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
                else launch_nw<128, 2>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
            } else {
                if (c->waves == 8) launch_nw<64, 8>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
                else if (c->waves == 4) launch_nw<64, 4>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
                else launch_nw<64, 2>(*c, Kl, Vl, lcap_blk, nblk, rev, sink, s);
            }
        };
        for (int i = 0; i < 2 * c->layers; ++i) run(i);  // warm-up
        const bool rec0 = hipEventRecord(e0, nullptr) == hipSuccess;
        for (int i = 0; i < c->launches; ++i) run(2 * c->layers + i);
        const bool rec1 = hipEventRecord(e1, nullptr) == hipSuccess;
        float ms = 0.f;
        if (rec0 && rec1 && hipEventSynchronize(e1) == hipSuccess && hipEventElapsedTime(&ms, e0, e1) == hipSuccess &&
            hipGetLastError() == hipSuccess) {
            *us_per_launch = 1e3 * ms / c->launches;
            *bytes_per_launch = (double)per_layer * 2 * 2;
            rc = 0;
        }
    }
    // release what was taken (a failure here leaves nothing more to undo)
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (K) (void)hipFree(K);
    if (V) (void)hipFree(V);
    if (sink) (void)hipFree(sink);
    return rc;
}
