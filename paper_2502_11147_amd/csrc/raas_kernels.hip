// gfx950 kernels of the page-based RaaS decode path (arXiv 2502.11147,
// Algorithm 1 and Sections 3.2-3.3).
//
// Pool layout in HBM, per unit (sequence, layer, KV head): a contiguous run of
// Lcap = roundup(S * page_size, 32) token rows for K and for V. Token t of
// slot s sits at row s * page_size + t. Rows are grouped in blocks of 32; in a
// bf16 pool each block is stored in the order the attention kernel's MFMA
// operands are loaded, so that every 16-byte-per-lane load of a wavefront
// reads 1 KiB of consecutive bytes:
//   K block: [2 row tiles][D/32 k-steps][4 lane groups][16 rows][8 channels],
//            tile q, row i holding token 8*(i/4) + 4*q + i%4, lane group a
//            channels 32*ks + 8*a .. +8;
//   V block: [D/16 channel tiles][4 token octets][16 channels][8 tokens],
//            i.e. V transposed so a lane reads 8 consecutive tokens of one
//            channel.
// An fp32 pool keeps plain [row][channel] order.
#include <math.h>

#include "raas_internal.h"

namespace raas {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }

// round to nearest even; inputs are finite
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t b = __float_as_uint(f);
    b += 0x7FFFu + ((b >> 16) & 1u);
    return (uint16_t)(b >> 16);
}

template <typename T>
__device__ __forceinline__ float to_f(T x);
template <>
__device__ __forceinline__ float to_f<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f<uint16_t>(uint16_t x) { return bf2f(x); }

template <typename T>
__device__ __forceinline__ T from_f(float x);
template <>
__device__ __forceinline__ float from_f<float>(float x) { return x; }
template <>
__device__ __forceinline__ uint16_t from_f<uint16_t>(float x) { return f2bf(x); }

// element offset of (token row t, channel c) inside a unit's bf16 K run
template <int D>
__device__ __forceinline__ size_t k_off(int t, int c) {
    const int b = t >> 5, tt = t & 31;
    const int i = 4 * (tt >> 3) + (tt & 3), qq = (tt >> 2) & 1;
    const int ks = c >> 5, a = (c >> 3) & 3, e = c & 7;
    return (size_t)b * 32 * D + (size_t)(qq * (D / 32) + ks) * 512 + (16 * a + i) * 8 + e;
}

// element offset of (token row t, channel c) inside a unit's bf16 V run
template <int D>
__device__ __forceinline__ size_t v_off(int t, int c) {
    const int b = t >> 5, tt = t & 31;
    const int nb = c >> 4, i = c & 15, a = tt >> 3, j = tt & 7;
    return (size_t)b * 32 * D + (size_t)nb * 512 + (16 * a + i) * 8 + j;
}

__device__ __forceinline__ bf16x8 ld_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// ---------------------------------------------------------------------------
// Prefill: store the first keep_tok tokens of every unit and mark pages
// 0..keep_pages-1 pinned (kvm.store_cache(.., "prefill"), Algorithm 1).

__global__ void k_prefill_meta(LayerView L, int P, int keep_pages) {
    const int u = blockIdx.x;
    const size_t base = (size_t)u * L.S;
    for (int s = threadIdx.x; s < L.S; s += blockDim.x) {
        const bool pin = s < keep_pages;
        L.state[base + s] = pin ? kPinned : kFree;
        L.lid[base + s] = pin ? s : -1;
        L.ts[base + s] = -1;
        L.fill[base + s] = pin ? min(L.ps, P - s * L.ps) : 0;
    }
    if (threadIdx.x == 0) {
        int32_t* U4 = L.unit + 4 * (size_t)u;
        U4[kTail] = -1;
        U4[kNextLid] = (P + L.ps - 1) / L.ps;
        U4[kClock] = P;
        U4[kEvicted] = -1;
    }
}

template <int D>
__global__ void k_prefill_bf16(LayerView L, const uint16_t* __restrict__ k,
                               const uint16_t* __restrict__ v, int P, int keep_tok) {
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t nK = (size_t)L.U * keep_tok * (D / 8);
    const int octets = (keep_tok + 7) / 8;
    const size_t nV = (size_t)L.U * octets * D;
    uint16_t* K = (uint16_t*)L.K;
    uint16_t* V = (uint16_t*)L.V;
    if (tid < nK) {
        const int u = (int)(tid / ((size_t)keep_tok * (D / 8)));
        const int rem = (int)(tid - (size_t)u * keep_tok * (D / 8));
        const int t = rem / (D / 8), ch = rem % (D / 8);
        const u32x4 x = *reinterpret_cast<const u32x4*>(k + ((size_t)u * P + t) * D + ch * 8);
        *reinterpret_cast<u32x4*>(K + (size_t)u * L.Lcap * D + k_off<D>(t, ch * 8)) = x;
    } else if (tid - nK < nV) {
        const size_t r = tid - nK;
        const int u = (int)(r / ((size_t)octets * D));
        const int rem = (int)(r - (size_t)u * octets * D);
        const int g = rem / D, c = rem % D;
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
            const int t0 = 8 * g + j, t1 = t0 + 1;
            const uint32_t lo = (t0 < keep_tok) ? v[((size_t)u * P + t0) * D + c] : 0u;
            const uint32_t hi = (t1 < keep_tok) ? v[((size_t)u * P + t1) * D + c] : 0u;
            w[j / 2] = lo | (hi << 16);
        }
        u32x4 x = {w[0], w[1], w[2], w[3]};
        *reinterpret_cast<u32x4*>(V + (size_t)u * L.Lcap * D + v_off<D>(8 * g, c)) = x;
    }
}

__global__ void k_prefill_f32(LayerView L, const float* __restrict__ k, const float* __restrict__ v,
                              int P, int keep_tok) {
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int D = L.D;
    const size_t n = (size_t)L.U * keep_tok * (D / 4);
    if (tid >= n) return;
    const int u = (int)(tid / ((size_t)keep_tok * (D / 4)));
    const int rem = (int)(tid - (size_t)u * keep_tok * (D / 4));
    const int t = rem / (D / 4), ch = rem % (D / 4);
    const size_t src = ((size_t)u * P + t) * D + ch * 4;
    const size_t dst = ((size_t)u * L.Lcap + t) * D + ch * 4;
    *reinterpret_cast<float4*>((float*)L.K + dst) = *reinterpret_cast<const float4*>(k + src);
    *reinterpret_cast<float4*>((float*)L.V + dst) = *reinterpret_cast<const float4*>(v + src);
}

// ---------------------------------------------------------------------------
// Append (Algorithm 1, "store K_new and V_new"; Section 3.3 pages): one
// wavefront per unit. When the tail page is full or absent the lowest free
// slot becomes a fresh evictable page stamped with the clock. Eviction at the
// end of the previous step guarantees a free slot in that case.

template <typename T, int D>
__global__ __launch_bounds__(64) void k_append(LayerView L, const T* __restrict__ k_new,
                                               const T* __restrict__ v_new) {
    const int u = blockIdx.x, lane = threadIdx.x;
    const int S = L.S, ps = L.ps;
    const size_t base = (size_t)u * S;
    int32_t* U4 = L.unit + 4 * (size_t)u;
    int tail = U4[kTail];
    int f = (tail >= 0) ? L.fill[base + tail] : ps;
    if (f == ps) {
        int s = -1;
        for (int b0 = 0; b0 < S; b0 += 64) {
            const int s_ = b0 + lane;
            const bool fr = (s_ < S) && L.state[base + s_] == kFree;
            const unsigned long long m = __ballot(fr);
            if (m) {
                s = b0 + __builtin_ctzll(m);
                break;
            }
        }
        if (s < 0) {  // cannot happen: the previous step evicted when full
            if (lane == 0) atomicOr(L.err, 1);
            return;
        }
        if (lane == 0) {
            const int nl = U4[kNextLid];
            L.state[base + s] = kEvictable;
            L.lid[base + s] = nl;
            L.ts[base + s] = U4[kClock];
            U4[kNextLid] = nl + 1;
            U4[kTail] = s;
        }
        tail = s;
        f = 0;
    }
    const T* kn = k_new + (size_t)u * D;
    const T* vn = v_new + (size_t)u * D;
    const int row = tail * ps + f;
    T* kmin = (T*)L.kmin + (base + tail) * D;
    T* kmax = (T*)L.kmax + (base + tail) * D;
    for (int c = lane; c < D; c += 64) {
        const T x = kn[c];
        if (f == 0) {
            kmin[c] = x;
            kmax[c] = x;
        } else {
            if (to_f<T>(x) < to_f<T>(kmin[c])) kmin[c] = x;
            if (to_f<T>(x) > to_f<T>(kmax[c])) kmax[c] = x;
        }
    }
    if constexpr (sizeof(T) == 2) {
        uint16_t* Ku = (uint16_t*)L.K + (size_t)u * L.Lcap * D;
        uint16_t* Vu = (uint16_t*)L.V + (size_t)u * L.Lcap * D;
        if (lane < D / 8)
            *reinterpret_cast<u32x4*>(Ku + k_off<D>(row, lane * 8)) =
                *reinterpret_cast<const u32x4*>((const uint16_t*)kn + lane * 8);
        for (int c = lane; c < D; c += 64) Vu[v_off<D>(row, c)] = ((const uint16_t*)vn)[c];
    } else {
        float* Ku = (float*)L.K + ((size_t)u * L.Lcap + row) * D;
        float* Vu = (float*)L.V + ((size_t)u * L.Lcap + row) * D;
        for (int c = lane; c < D; c += 64) {
            Ku[c] = (float)kn[c];
            Vu[c] = (float)vn[c];
        }
    }
    if (lane == 0) L.fill[base + tail] = f + 1;
}

// ---------------------------------------------------------------------------
// Attention over every resident token (Algorithm 1, attention(Q, K_old::K_new,
// V_old::V_new)), split-K over 32-token blocks.
//
// bf16 pools: one workgroup of kAttnWaves wavefronts per (unit, split); each
// wavefront holds the unit's whole GQA query group and walks blocks
// round-robin. Per block: QK^T as two 16x16x32 bf16 MFMA tiles per 32
// channels (rows = tokens, columns = query heads, G <= 16 of the 16 used),
// online softmax in base 2 with one cross-lane max per block, and PV as
// D/16 MFMAs of V^T (rows = channels) times P^T (columns = heads). A lane
// owns one head (its column) in both products, so no data moves between
// lanes except the block max. Partial (max, sum, acc) of the wavefronts are
// merged through LDS; with several splits the workgroup writes a partial
// that k_merge combines.

template <int D>
__global__ __launch_bounds__(kAttnWaves * 64) void k_attn_bf16(LayerView L, const uint16_t* __restrict__ q,
                                                           float* __restrict__ part,
                                                           uint16_t* __restrict__ out, int nsplit,
                                                           int bps, float scale_log2) {
    constexpr int KS = D / 32, NB = D / 16, BLK = 32 * D;
    __shared__ float s_m[kAttnWaves][16];
    __shared__ float s_l[kAttnWaves][16];
    __shared__ __align__(16) float s_o[kAttnWaves][16][D + 4];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int grp = lane >> 4, col = lane & 15;
    const int u = blockIdx.x / nsplit, split = blockIdx.x - (blockIdx.x / nsplit) * nsplit;
    const int G = L.G, S = L.S, ps = L.ps;
    const int nblk = L.Lcap / 32;
    const int b0 = split * bps;
    const int b1 = min(nblk, b0 + bps);
    const uint16_t* Ku = (const uint16_t*)L.K + (size_t)u * L.Lcap * D;
    const uint16_t* Vu = (const uint16_t*)L.V + (size_t)u * L.Lcap * D;
    const int32_t* fu = L.fill + (size_t)u * S;

    bf16x8 qv[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if (col < G) {
            qv[ks] = ld_bf16x8(q + ((size_t)u * G + col) * D + 32 * ks + 8 * grp);
        } else {
            qv[ks] = __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u});
        }
    }
    float m_run = -INFINITY, l_run = 0.0f;
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int b = b0 + w; b < b1; b += kAttnWaves) {
        // tokens 8*grp .. 8*grp+7 of the block lie in one page (page_size % 8 == 0)
        const int t0 = 32 * b + 8 * grp;
        const int slot = t0 / ps;
        const int pos0 = t0 - slot * ps;
        const int f = (slot < S) ? fu[slot] : 0;
        const int nv = min(max(f - pos0, 0), 8);
        if (__ballot(nv > 0) == 0ull) continue;

        const uint16_t* Kb = Ku + (size_t)b * BLK + lane * 8;
        const uint16_t* Vb = Vu + (size_t)b * BLK + lane * 8;
        bf16x8 kr[2][KS], vr[NB];
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kr[qq][ks] = ld_bf16x8(Kb + (qq * KS + ks) * 512);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) vr[nb] = ld_bf16x8(Vb + nb * 512);

        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[0][ks], qv[ks], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kr[1][ks], qv[ks], s1, 0, 0, 0);
        }
        // x[j]: scaled logit of token 8*grp + j for head `col` (base 2)
        float x[8];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            x[v] = (v < nv) ? s0[v] * scale_log2 : -INFINITY;
            x[4 + v] = (4 + v < nv) ? s1[v] * scale_log2 : -INFINITY;
        }
        float mb = x[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) mb = fmaxf(mb, x[j]);
        mb = fmaxf(mb, __shfl_xor(mb, 16));
        mb = fmaxf(mb, __shfl_xor(mb, 32));
        const float m_new = fmaxf(m_run, mb);
        if (__ballot(m_new > m_run) != 0ull) {
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            l_run *= alpha;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] *= alpha;
            m_run = m_new;
        }
        float p[8], psum = 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            p[j] = __builtin_amdgcn_exp2f(x[j] - m_run);
            psum += p[j];
        }
        l_run += psum;
        bf16x8 pb;
#pragma unroll
        for (int j = 0; j < 8; ++j) pb[j] = (__bf16)p[j];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vr[nb], pb, acc[nb], 0, 0, 0);
    }

    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (grp == 0) {
        s_m[w][col] = m_run;
        s_l[w][col] = l_run;
    }
    if (col < G) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            *reinterpret_cast<f32x4*>(&s_o[w][col][16 * nb + 4 * grp]) = acc[nb];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < G * D; idx += kAttnWaves * 64) {
        const int h = idx / D, c = idx - (idx / D) * D;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kAttnWaves; ++ww) M = fmaxf(M, s_m[ww][h]);
        float O = 0.0f, Ls = 0.0f;
#pragma unroll
        for (int ww = 0; ww < kAttnWaves; ++ww) {
            const float mw = s_m[ww][h];
            const float wt = (mw == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mw - M);
            O += wt * s_o[ww][h][c];
            Ls += wt * s_l[ww][h];
        }
        if (nsplit == 1) {
            out[((size_t)u * G + h) * D + c] = f2bf(O / Ls);
        } else {
            float* pp = part + (((size_t)u * nsplit + split) * G + h) * (D + 2);
            pp[c] = O;
            if (c == 0) {
                pp[D] = M;
                pp[D + 1] = Ls;
            }
        }
    }
}

// fp32 pools: one wavefront per (unit, split), one token at a time, lanes
// across channels; online softmax per head in fp32.
template <int D>
__global__ __launch_bounds__(64) void k_attn_f32(LayerView L, const float* __restrict__ q,
                                                 float* __restrict__ part, float* __restrict__ out,
                                                 int nsplit, int tps, float scale_log2) {
    constexpr int DPL = D / 64;
    const int lane = threadIdx.x;
    const int u = blockIdx.x / nsplit, split = blockIdx.x - (blockIdx.x / nsplit) * nsplit;
    const int G = L.G, S = L.S, ps = L.ps;
    const int t0 = split * tps;
    const int t1 = min(S * ps, t0 + tps);
    const float* Ku = (const float*)L.K + (size_t)u * L.Lcap * D;
    const float* Vu = (const float*)L.V + (size_t)u * L.Lcap * D;
    const int32_t* fu = L.fill + (size_t)u * S;

    float qr[16][DPL], m[16], l[16], acc[16][DPL];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        m[j] = -INFINITY;
        l[j] = 0.0f;
#pragma unroll
        for (int i = 0; i < DPL; ++i) {
            qr[j][i] = (j < G) ? q[((size_t)u * G + j) * D + lane + 64 * i] : 0.0f;
            acc[j][i] = 0.0f;
        }
    }
    for (int t = t0; t < t1; ++t) {
        const int slot = t / ps;
        if (t - slot * ps >= fu[slot]) continue;
        float kr[DPL], vr[DPL];
#pragma unroll
        for (int i = 0; i < DPL; ++i) {
            kr[i] = Ku[(size_t)t * D + lane + 64 * i];
            vr[i] = Vu[(size_t)t * D + lane + 64 * i];
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            if (j >= G) break;
            float dot = 0.0f;
#pragma unroll
            for (int i = 0; i < DPL; ++i) dot = fmaf(qr[j][i], kr[i], dot);
            const float x = wave_sum(dot) * scale_log2;
            const float m_new = fmaxf(m[j], x);
            const float alpha = __builtin_amdgcn_exp2f(m[j] - m_new);
            const float p = __builtin_amdgcn_exp2f(x - m_new);
            l[j] = l[j] * alpha + p;
#pragma unroll
            for (int i = 0; i < DPL; ++i) acc[j][i] = fmaf(p, vr[i], acc[j][i] * alpha);
            m[j] = m_new;
        }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        if (j >= G) break;
        if (nsplit == 1) {
#pragma unroll
            for (int i = 0; i < DPL; ++i) out[((size_t)u * G + j) * D + lane + 64 * i] = acc[j][i] / l[j];
        } else {
            float* pp = part + (((size_t)u * nsplit + split) * G + j) * (D + 2);
#pragma unroll
            for (int i = 0; i < DPL; ++i) pp[lane + 64 * i] = acc[j][i];
            if (lane == 0) {
                pp[D] = m[j];
                pp[D + 1] = l[j];
            }
        }
    }
}

// Split-K merge: out = sum_s 2^(M_s - M) O_s / sum_s 2^(M_s - M) L_s.
template <typename T>
__global__ __launch_bounds__(256) void k_merge(LayerView L, const float* __restrict__ part,
                                               T* __restrict__ out, int nsplit) {
    const int u = blockIdx.x, G = L.G, D = L.D;
    for (int idx = threadIdx.x; idx < G * D; idx += blockDim.x) {
        const int h = idx / D, c = idx - (idx / D) * D;
        float M = -INFINITY;
        for (int s = 0; s < nsplit; ++s)
            M = fmaxf(M, part[(((size_t)u * nsplit + s) * G + h) * (D + 2) + D]);
        float O = 0.0f, Ls = 0.0f;
        for (int s = 0; s < nsplit; ++s) {
            const float* pp = part + (((size_t)u * nsplit + s) * G + h) * (D + 2);
            const float ms = pp[D];
            const float wt = (ms == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(ms - M);
            O += wt * pp[c];
            Ls += wt * pp[D + 1];
        }
        out[((size_t)u * G + h) * D + c] = from_f<T>(O / Ls);
    }
}

// ---------------------------------------------------------------------------
// Score, threshold, refresh, evict (Algorithm 1, store_cache; Sections
// 3.2-3.3): one workgroup per unit.
//  - Each evictable page gets max over the G query heads of
//    sum_c max(q_c*kmax_c, q_c*kmin_c), accumulated in fp64 (products of
//    bf16 or fp32 values are exact in fp64); 16 lanes per page, each summing
//    D/16 channels in order, then a fixed xor tree, so equal pages score
//    equal.
//  - With n evictable pages and k = floor(r*n), page p is refreshed (ts =
//    clock) when at least n-k evictable pages score strictly less than it:
//    exactly the pages above the (n-k)-th smallest score.
//  - When the tail page is full and no slot is free, the evictable page with
//    the smallest (timestamp, logical id) is freed.
template <typename T, int D>
__global__ __launch_bounds__(256) void k_score(LayerView L, const T* __restrict__ q, StepIO io,
                                               double r) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int S = L.S, G = L.G;
    double* s_q = reinterpret_cast<double*>(smem);  // [G][D]
    double* s_score = s_q + (size_t)G * D;          // [S]
    int* s_ts = reinterpret_cast<int*>(s_score + S); // [S]
    int* s_state = s_ts + S;                        // [S]
    __shared__ int s_cnt[2];
    __shared__ unsigned long long s_min;
    __shared__ int s_victim;

    const int u = blockIdx.x, tid = threadIdx.x;
    const size_t base = (size_t)u * S;
    int32_t* U4 = L.unit + 4 * (size_t)u;
    const int clock = U4[kClock];
    for (int i = tid; i < G * D; i += 256) s_q[i] = (double)to_f<T>(q[(size_t)u * G * D + i]);
    for (int s = tid; s < S; s += 256) {
        s_state[s] = L.state[base + s];
        s_ts[s] = L.ts[base + s];
    }
    if (tid == 0) {
        s_cnt[0] = 0;
        s_cnt[1] = 0;
        s_min = ~0ull;
        s_victim = -1;
    }
    __syncthreads();

    constexpr int DPL = D / 16;
    const int g = tid >> 4, li = tid & 15;
    const T* kmax_u = (const T*)L.kmax + base * D;
    const T* kmin_u = (const T*)L.kmin + base * D;
    for (int p0 = 0; p0 < S; p0 += 16) {
        const int p = p0 + g;
        const bool act = (p < S) && s_state[p] == kEvictable;
        double kx[DPL], kn[DPL];
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            kx[e] = act ? (double)to_f<T>(kmax_u[(size_t)p * D + li * DPL + e]) : 0.0;
            kn[e] = act ? (double)to_f<T>(kmin_u[(size_t)p * D + li * DPL + e]) : 0.0;
        }
        double best = -INFINITY;
        for (int j = 0; j < G; ++j) {
            const double* qj = s_q + (size_t)j * D + li * DPL;
            double a = 0.0;
#pragma unroll
            for (int e = 0; e < DPL; ++e) {
                const double hi = qj[e] * kx[e];
                const double lo = qj[e] * kn[e];
                a += (hi > lo) ? hi : lo;
            }
            a += __shfl_xor(a, 8);
            a += __shfl_xor(a, 4);
            a += __shfl_xor(a, 2);
            a += __shfl_xor(a, 1);
            best = (a > best) ? a : best;
        }
        if (act && li == 0) s_score[p] = best;
    }
    int ev = 0, fr = 0;
    for (int s = tid; s < S; s += 256) {
        ev += (s_state[s] == kEvictable);
        fr += (s_state[s] == kFree);
    }
    if (ev) atomicAdd(&s_cnt[0], ev);
    if (fr) atomicAdd(&s_cnt[1], fr);
    __syncthreads();

    const int n = s_cnt[0], nfree = s_cnt[1];
    const int k = (int)floor(r * (double)n);
    if (k > 0) {
        for (int p = tid; p < S; p += 256) {
            if (s_state[p] != kEvictable) continue;
            const double sp = s_score[p];
            int less = 0;
            for (int o = 0; o < S; ++o) less += (s_state[o] == kEvictable && s_score[o] < sp);
            if (less >= n - k) s_ts[p] = clock;
        }
    }
    __syncthreads();

    const int tail = U4[kTail];
    const bool full = tail >= 0 && L.fill[base + tail] == L.ps && nfree == 0;
    int evicted = -1;
    if (full) {
        unsigned long long best = ~0ull;
        for (int s = tid; s < S; s += 256) {
            if (s_state[s] != kEvictable) continue;
            const unsigned long long key =
                ((unsigned long long)(uint32_t)s_ts[s] << 32) | (uint32_t)L.lid[base + s];
            best = key < best ? key : best;
        }
        if (best != ~0ull) atomicMin(&s_min, best);
        __syncthreads();
        for (int s = tid; s < S; s += 256) {
            if (s_state[s] != kEvictable) continue;
            const unsigned long long key =
                ((unsigned long long)(uint32_t)s_ts[s] << 32) | (uint32_t)L.lid[base + s];
            if (key == s_min) s_victim = s;
        }
        __syncthreads();
        const int v = s_victim;
        if (v >= 0) {
            evicted = (int)(s_min & 0xFFFFFFFFull);
            if (tid == 0) {
                s_state[v] = kFree;
                s_ts[v] = -1;
            }
        } else if (tid == 0) {
            atomicOr(L.err, 2);
        }
        __syncthreads();
        if (v >= 0 && tid == 0) {
            L.lid[base + v] = -1;
            L.fill[base + v] = 0;
            if (tail == v) U4[kTail] = -1;
        }
    }
    for (int s = tid; s < S; s += 256) {
        L.ts[base + s] = s_ts[s];
        L.state[base + s] = s_state[s];
        if (io.page_table_out)
            io.page_table_out[base + s] = (s_state[s] == kFree) ? -1 : L.lid[base + s];
        if (io.timestamps_out) io.timestamps_out[base + s] = (s_state[s] == kEvictable) ? s_ts[s] : -1;
    }
    if (tid == 0) {
        U4[kClock] = clock + 1;
        U4[kEvicted] = evicted;
        if (io.evicted_out) io.evicted_out[u] = evicted;
    }
}

inline unsigned grid1d(size_t n, int block) { return (unsigned)((n + block - 1) / block); }

}  // namespace

// ---------------------------------------------------------------------------
// launchers

hipError_t launch_prefill(const LayerView& L, const void* k, const void* v, int P, int keep_pages,
                          hipStream_t stream) {
    hipLaunchKernelGGL(k_prefill_meta, dim3(L.U), dim3(256), 0, stream, L, P, keep_pages);
    const int keep_tok = min(P, keep_pages * L.ps);
    if (keep_tok > 0) {
        if (L.bf16) {
            const size_t n = (size_t)L.U * keep_tok * (L.D / 8) + (size_t)L.U * ((keep_tok + 7) / 8) * L.D;
            if (L.D == 128)
                hipLaunchKernelGGL(k_prefill_bf16<128>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const uint16_t*)k, (const uint16_t*)v, P, keep_tok);
            else
                hipLaunchKernelGGL(k_prefill_bf16<64>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const uint16_t*)k, (const uint16_t*)v, P, keep_tok);
        } else {
            const size_t n = (size_t)L.U * keep_tok * (L.D / 4);
            hipLaunchKernelGGL(k_prefill_f32, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                               (const float*)k, (const float*)v, P, keep_tok);
        }
    }
    return hipGetLastError();
}

hipError_t launch_append(const LayerView& L, const StepIO& io, hipStream_t stream) {
    if (L.bf16) {
        if (L.D == 128)
            hipLaunchKernelGGL((k_append<uint16_t, 128>), dim3(L.U), dim3(64), 0, stream, L,
                               (const uint16_t*)io.k_new, (const uint16_t*)io.v_new);
        else
            hipLaunchKernelGGL((k_append<uint16_t, 64>), dim3(L.U), dim3(64), 0, stream, L,
                               (const uint16_t*)io.k_new, (const uint16_t*)io.v_new);
    } else {
        if (L.D == 128)
            hipLaunchKernelGGL((k_append<float, 128>), dim3(L.U), dim3(64), 0, stream, L,
                               (const float*)io.k_new, (const float*)io.v_new);
        else
            hipLaunchKernelGGL((k_append<float, 64>), dim3(L.U), dim3(64), 0, stream, L,
                               (const float*)io.k_new, (const float*)io.v_new);
    }
    return hipGetLastError();
}

hipError_t launch_attention(const LayerView& L, const StepIO& io, int nsplit, int bps,
                            float* partials, hipStream_t stream) {
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)L.D));
    const dim3 grid((unsigned)(L.U * nsplit));
    if (L.bf16) {
        if (L.D == 128)
            hipLaunchKernelGGL(k_attn_bf16<128>, grid, dim3(kAttnWaves * 64), 0, stream, L,
                               (const uint16_t*)io.q, partials, (uint16_t*)io.out, nsplit, bps, scale_log2);
        else
            hipLaunchKernelGGL(k_attn_bf16<64>, grid, dim3(kAttnWaves * 64), 0, stream, L,
                               (const uint16_t*)io.q, partials, (uint16_t*)io.out, nsplit, bps, scale_log2);
    } else {
        const int tps = bps * 32;
        if (L.D == 128)
            hipLaunchKernelGGL(k_attn_f32<128>, grid, dim3(64), 0, stream, L, (const float*)io.q,
                               partials, (float*)io.out, nsplit, tps, scale_log2);
        else
            hipLaunchKernelGGL(k_attn_f32<64>, grid, dim3(64), 0, stream, L, (const float*)io.q,
                               partials, (float*)io.out, nsplit, tps, scale_log2);
    }
    return hipGetLastError();
}

hipError_t launch_merge(const LayerView& L, const StepIO& io, int nsplit, const float* partials,
                        hipStream_t stream) {
    if (L.bf16)
        hipLaunchKernelGGL(k_merge<uint16_t>, dim3(L.U), dim3(256), 0, stream, L, partials,
                           (uint16_t*)io.out, nsplit);
    else
        hipLaunchKernelGGL(k_merge<float>, dim3(L.U), dim3(256), 0, stream, L, partials,
                           (float*)io.out, nsplit);
    return hipGetLastError();
}

hipError_t launch_score(const LayerView& L, const StepIO& io, double r, hipStream_t stream) {
    const size_t shm = (size_t)L.G * L.D * sizeof(double) + (size_t)L.S * (sizeof(double) + 2 * sizeof(int));
    if (L.bf16) {
        if (L.D == 128)
            hipLaunchKernelGGL((k_score<uint16_t, 128>), dim3(L.U), dim3(256), shm, stream, L,
                               (const uint16_t*)io.q, io, r);
        else
            hipLaunchKernelGGL((k_score<uint16_t, 64>), dim3(L.U), dim3(256), shm, stream, L,
                               (const uint16_t*)io.q, io, r);
    } else {
        if (L.D == 128)
            hipLaunchKernelGGL((k_score<float, 128>), dim3(L.U), dim3(256), shm, stream, L,
                               (const float*)io.q, io, r);
        else
            hipLaunchKernelGGL((k_score<float, 64>), dim3(L.U), dim3(256), shm, stream, L,
                               (const float*)io.q, io, r);
    }
    return hipGetLastError();
}

}  // namespace raas
