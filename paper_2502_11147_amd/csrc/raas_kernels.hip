// gfx950 kernels of the page-based RaaS decode path (arXiv 2502.11147,
// Algorithm 1 and Sections 3.2-3.3).
//
// Pool layout in HBM, per unit (sequence, layer, KV head): a contiguous run of
// Lcap = roundup(S * page_size, 32) token rows for K and for V. Token t of
// slot s sits at row s * page_size + t. Rows are grouped in blocks of 32; in a
// bf16 pool each block is stored in the order the attention MFMA operands
// are loaded, so that every 16-byte-per-lane load of a wavefront reads 1 KiB
// of consecutive bytes:
//   K block: [2 row tiles][D/32 k-steps][4 lane groups][16 rows][8 channels],
//            tile q, row i holding token 8*(i/4) + 4*q + i%4, lane group a
//            channels 32*ks + 8*a .. +8;
//   V block: [D/16 channel tiles][4 token octets][16 channels][8 tokens],
//            V transposed so a lane reads 8 consecutive tokens of one channel.
// An fp32 pool keeps plain [row][channel] order.
//
// One decode step is one launch of a step kernel (attention over the
// resident pages with the new token substituted in registers, the append of
// that token, the page scores) whose workgroup, when one workgroup covers a
// whole unit, also runs the epilogue (top-r refresh, eviction, next target
// slot, state out). When a unit is split over several workgroups, or the pool
// is fp32, the epilogue is a second kernel that also merges the splits.
#include <math.h>

#include <algorithm>
#include <utility>

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

__device__ __forceinline__ u32x4 ld4(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st4(void* p, u32x4 x) { *reinterpret_cast<u32x4*>(p) = x; }

__device__ __forceinline__ uint16_t u16_at(const u32x4& x, int e) {
    return (uint16_t)((x[e >> 1] >> ((e & 1) * 16)) & 0xFFFFu);
}

// ---------------------------------------------------------------------------
// Prefill (the prefill stage of Algorithm 1's cache store): a unit's first
// tokens go to pages 0, 1, ..., which are marked pinned; at most S-1 pages
// are kept (the first ones), so one slot stays for decode pages. Lengths are
// per sequence (in.lens) or uniform (in.P); in.mask, when given, selects the
// sequences to (re)initialise and leaves the others as they are. The input
// holds in.stride rows per unit.

// Prefill length of unit u, or -1 when its sequence is not selected.
__device__ __forceinline__ int unit_prefill_len(const LayerView& L, const PrefillIn& in, int u) {
    const int seq = u / L.nkv;
    if (in.mask != nullptr && in.mask[seq] == 0) return -1;
    return in.lens != nullptr ? in.lens[seq] : in.P;
}

// pages kept of a prefill of P tokens: the first min(ceil(P/ps), pcap)
// (pcap = S-1, or the prompt region's slots)
__device__ __forceinline__ int kept_pages(const LayerView& L, int P) {
    return min((P + L.ps - 1) / L.ps, L.pcap);
}

__global__ void k_prefill_meta(LayerView L, PrefillIn in) {
    const int u = blockIdx.x;
    const int P = unit_prefill_len(L, in, u);
    if (P < 0) return;
    const int keep_pages = kept_pages(L, P);
    const size_t base = (size_t)u * L.S;
    for (int s = threadIdx.x; s < L.S; s += blockDim.x) {
        const bool pin = s < keep_pages;
        L.state[base + s] = pin ? kPinned : kFree;
        L.lid[base + s] = pin ? s : -1;
        L.ts[base + s] = -1;
        L.fill[base + s] = pin ? min(L.ps, P - s * L.ps) : 0;
    }
    if (threadIdx.x == 0) {
        int32_t* U4 = L.unit + (size_t)u * kUnitFields;
        U4[kTail] = -1;
        U4[kNextLid] = (P + L.ps - 1) / L.ps;
        U4[kClock] = P;
        U4[kEvicted] = -1;
        U4[kNextSlot] = max(keep_pages, L.dbase);  // lowest free decode slot; decode starts a fresh page
        U4[kNextFill] = 0;
        U4[kPinnedPages] = keep_pages;
    }
}

// K rows (D/8 threads per token) then V octets (D threads per 8 tokens),
// over max_tok tokens per unit; tokens past a unit's kept ones are skipped
// (K) or zero (the rest of V's last octet).
template <int D>
__global__ void k_prefill_bf16(LayerView L, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
                               PrefillIn in, int max_tok) {
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const size_t nK = (size_t)L.U * max_tok * (D / 8);
    const int octets = (max_tok + 7) / 8;
    const size_t nV = (size_t)L.U * octets * D;
    uint16_t* K = (uint16_t*)L.K;
    uint16_t* V = (uint16_t*)L.V;
    if (tid < nK) {
        const int u = (int)(tid / ((size_t)max_tok * (D / 8)));
        const int rem = (int)(tid - (size_t)u * max_tok * (D / 8));
        const int t = rem / (D / 8), ch = rem % (D / 8);
        const int P = unit_prefill_len(L, in, u);
        if (t >= min(P, kept_pages(L, P) * L.ps)) return;  // also P < 0: not selected
        st4(K + (size_t)u * L.Lcap * D + k_off<D>(t, ch * 8), ld4(k + ((size_t)u * in.stride + t) * D + ch * 8));
    } else if (tid - nK < nV) {
        const size_t r = tid - nK;
        const int u = (int)(r / ((size_t)octets * D));
        const int rem = (int)(r - (size_t)u * octets * D);
        const int g = rem / D, c = rem % D;
        const int P = unit_prefill_len(L, in, u);
        const int keep_tok = min(P, kept_pages(L, P) * L.ps);
        if (8 * g >= keep_tok) return;
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 8; j += 2) {
            const int t0 = 8 * g + j, t1 = t0 + 1;
            const uint32_t lo = (t0 < keep_tok) ? v[((size_t)u * in.stride + t0) * D + c] : 0u;
            const uint32_t hi = (t1 < keep_tok) ? v[((size_t)u * in.stride + t1) * D + c] : 0u;
            w[j / 2] = lo | (hi << 16);
        }
        st4(V + (size_t)u * L.Lcap * D + v_off<D>(8 * g, c), u32x4{w[0], w[1], w[2], w[3]});
    }
}

__global__ void k_prefill_f32(LayerView L, const float* __restrict__ k, const float* __restrict__ v, PrefillIn in,
                              int max_tok) {
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int D = L.D;
    const size_t n = (size_t)L.U * max_tok * (D / 4);
    if (tid >= n) return;
    const int u = (int)(tid / ((size_t)max_tok * (D / 4)));
    const int rem = (int)(tid - (size_t)u * max_tok * (D / 4));
    const int t = rem / (D / 4), ch = rem % (D / 4);
    const int P = unit_prefill_len(L, in, u);
    if (t >= min(P, kept_pages(L, P) * L.ps)) return;
    const size_t src = ((size_t)u * in.stride + t) * D + ch * 4;
    const size_t dst = ((size_t)u * L.Lcap + t) * D + ch * 4;
    st4((float*)L.K + dst, ld4(k + src));
    st4((float*)L.V + dst, ld4(v + src));
}

// Representative keys of the pinned pages, needed only when they are ranked:
// per-channel min and max over each page's prefill tokens (Section 3.3). One
// thread per (unit, page, channel) over max_pages pages per unit; a
// wavefront reads 64 consecutive channels of one token at a time.
template <typename T>
__global__ void k_prefill_rep(LayerView L, const T* __restrict__ k, PrefillIn in, int max_pages) {
    const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int D = L.D, ps = L.ps;
    if (tid >= (size_t)L.U * max_pages * D) return;
    const int c = (int)(tid % D);
    const size_t up = tid / D;
    const int pg = (int)(up % max_pages), u = (int)(up / max_pages);
    const int P = unit_prefill_len(L, in, u);
    if (pg >= kept_pages(L, P)) return;            // also P < 0; else pg * ps < P
    const int t0 = pg * ps, t1 = min(P, t0 + ps);
    const T* ku = k + (size_t)u * in.stride * D + c;
    T hi = ku[(size_t)t0 * D], lo = hi;
    for (int t = t0 + 1; t < t1; ++t) {
        const T x = ku[(size_t)t * D];
        if (to_f(x) > to_f(hi)) hi = x;
        if (to_f(x) < to_f(lo)) lo = x;
    }
    const size_t o = ((size_t)u * L.S + pg) * D + c;
    ((T*)L.kmax)[o] = hi;
    ((T*)L.kmin)[o] = lo;
}

// ---------------------------------------------------------------------------
// Epilogue of a step, for one unit, run by every thread of one workgroup.
// Slot state is in LDS with the page the step opened already marked
// evictable; s_score holds the score of every evictable page.
//  - Top-r refresh (Algorithm 1; Section 3.2): with n evictable pages and
//    k = floor(r*n), page p gets ts = clock when at least n-k evictable
//    pages score strictly less, i.e. exactly the pages above the (n-k)-th
//    smallest score.
//  - Eviction (Algorithm 1, the eviction branch of the decode-stage store):
//    when the tail page is full and no slot is free, the evictable page
//    with the smallest (timestamp, logical id) is freed.
//  - The next token's target: the tail page if it has room, else the lowest
//    free slot (a fresh page).

// The unit record as read once at the start of a step.
struct UnitRec {
    int ns, nf, clock, next_lid;
    __device__ bool opened() const { return nf == 0; }
};

// Slots that take part in the top-r order statistic: the evictable pages,
// and the pinned ones when the pool ranks them.
__device__ __forceinline__ bool ranked(const LayerView& L, int st) {
    return st == kEvictable || (L.rank_pinned && st == kPinned);
}

__device__ __forceinline__ UnitRec read_unit(const LayerView& L, int u) {
    const int32_t* U4 = L.unit + (size_t)u * kUnitFields;
    return UnitRec{U4[kNextSlot], U4[kNextFill], U4[kClock], U4[kNextLid]};
}

// Stages slot s (state, timestamp, logical id as read from the pool) in LDS,
// with the page the step opens already marked evictable.
__device__ __forceinline__ void stage_slot(const UnitRec& ur, int s, int st, int t, int id, double* s_score,
                                           int* s_state, int* s_ts, int* s_lid) {
    if (s == ur.ns && ur.opened()) {
        st = kEvictable;
        t = ur.clock;
        id = ur.next_lid;
    }
    s_state[s] = st;
    s_ts[s] = t;
    s_lid[s] = id;
    s_score[s] = INFINITY;  // scored below when evictable; never ranks under a real score
}

__device__ void load_slots(const LayerView& L, int u, const UnitRec& ur, double* s_score, int* s_state,
                           int* s_ts, int* s_lid, int first = 0) {
    const int S = L.S;
    const size_t base = (size_t)u * S;
    for (int s = threadIdx.x + first; s < S; s += blockDim.x)
        stage_slot(ur, s, L.state[base + s], L.ts[base + s], L.lid[base + s], s_score, s_state, s_ts, s_lid);
}

// ---------------------------------------------------------------------------
// Page scores (Section 3.3, Quest's representative keys): for each evictable
// page, max over the G query heads of sum_c max(q_c*kmax_c, q_c*kmin_c),
// summed in fp64. A product of two bf16 values has at most 16 significant
// bits, so both products are formed exactly in fp32 (q and the keys are
// staged as fp32), the larger is widened and added in fp64: each add rounds
// exactly as the fp64 sum of the exact product (products below fp32's normal
// range, under 1e-38 in magnitude, would be the exception). Eight
// lanes per page: lane part p sums D/8 consecutive channels in two chains
// (even and odd channels), the eight parts combine through a fixed xor tree,
// so equal pages score equal. A wavefront scores 8 pages per pass; its passes
// are interleaved with its attention blocks, each pass's keys loading while
// the previous block computes. The page the step writes to has its min/max
// widened by the new key and stored back.

// Cross-lane moves that stay in the VALU (no LDS round trip). dpp_f64<CTRL>:
// a DPP move of both halves of a double; 0xB1 and 0x4E (quad_perm
// [1,0,3,2] and [2,3,0,1]) give lane ^ 1 and lane ^ 2, 0x141 (row_half_mirror)
// gives lane 7 - i within each group of 8. max_xor16_32: the max over lanes
// i, i ^ 16, i ^ 32 and i ^ 48 through the two permlane swaps (a swap of a
// value with itself leaves both 16-lane or 32-lane halves side by side).
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
    const unsigned long long b = __builtin_bit_cast(unsigned long long, x);
    const unsigned lo = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)b, CTRL, 0xF, 0xF, false);
    const unsigned hi = (unsigned)__builtin_amdgcn_update_dpp(0, (int)(unsigned)(b >> 32), CTRL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}
__device__ __forceinline__ float max_xor16_32(float x) {
    const unsigned u = __builtin_bit_cast(unsigned, x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float m = fmaxf(__builtin_bit_cast(float, (unsigned)a[0]), __builtin_bit_cast(float, (unsigned)a[1]));
    const unsigned v = __builtin_bit_cast(unsigned, m);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return fmaxf(__builtin_bit_cast(float, (unsigned)b[0]), __builtin_bit_cast(float, (unsigned)b[1]));
}
// Whole-wavefront max and sum of a float with no LDS round trip: lane ^ 1
// and lane ^ 2 by quad permutes, then the mirrors within 8 and within 16
// lanes (every lane of a quad, then of an 8-lane half, holds the same value
// by then), then the two permlane swaps. Every lane ends with the result,
// the sum in the same order on every lane.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_max_dpp(float x) {
    x = fmaxf(x, dpp_f32<0xB1>(x));
    x = fmaxf(x, dpp_f32<0x4E>(x));
    x = fmaxf(x, dpp_f32<0x141>(x));
    x = fmaxf(x, dpp_f32<0x140>(x));
    return max_xor16_32(x);
}
__device__ __forceinline__ float wave_sum_dpp(float x) {
    x += dpp_f32<0xB1>(x);
    x += dpp_f32<0x4E>(x);
    x += dpp_f32<0x141>(x);
    x += dpp_f32<0x140>(x);
    const unsigned u = __builtin_bit_cast(unsigned, x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    x = __builtin_bit_cast(float, (unsigned)a[0]) + __builtin_bit_cast(float, (unsigned)a[1]);
    const unsigned v = __builtin_bit_cast(unsigned, x);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __builtin_bit_cast(float, (unsigned)b[0]) + __builtin_bit_cast(float, (unsigned)b[1]);
}

// LDS slot of element i = head * D + channel of the fp32 query array: a
// 16-byte pad after each D/8 channels, so that the eight lanes scoring a
// page, which read channels D/8 apart, fall on different LDS banks and every
// group of four stays 16-byte aligned.
constexpr int qpad_row(int D) { return D + 32; }
template <int D>
__device__ __forceinline__ int qpad_index(int i) {
    const int h = i / D, c = i - (i / D) * D;
    return h * qpad_row(D) + c + 4 * (c / (D / 8));
}

template <int D>
struct ScoreFrag {
    static constexpr int SV = D / 64;  // 16-byte vectors per array per lane (D/8 bf16 channels)
    u32x4 kx[SV], kn[SV];
};

template <int D>
__device__ __forceinline__ void score_issue(const LayerView& L, int u, int p, int part, bool load,
                                            ScoreFrag<D>& f) {
    const size_t off = ((size_t)u * L.S + p) * D + part * (D / 8);
    const uint16_t* kx = (const uint16_t*)L.kmax + off;
    const uint16_t* kn = (const uint16_t*)L.kmin + off;
#pragma unroll
    for (int i = 0; i < ScoreFrag<D>::SV; ++i) {
        f.kx[i] = load ? ld4(kx + 8 * i) : u32x4{0u, 0u, 0u, 0u};
        f.kn[i] = load ? ld4(kn + 8 * i) : u32x4{0u, 0u, 0u, 0u};
    }
}

template <int D>
__device__ __forceinline__ double score_finish(const LayerView& L, int u, int p, int part, bool act,
                                               ScoreFrag<D>& f, bool is_tail, bool opened,
                                               const uint16_t* k_new, const float* qf, double* hb) {
    constexpr int SV = ScoreFrag<D>::SV;
    const int G = L.G;
    if (act && is_tail) {
#pragma unroll
        for (int i = 0; i < SV; ++i) {
            const u32x4 x = ld4(k_new + part * (D / 8) + 8 * i);
            if (opened) {
                f.kx[i] = x;
                f.kn[i] = x;
            } else {
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    uint32_t a = 0, b = 0;
#pragma unroll
                    for (int half = 0; half < 2; ++half) {
                        const uint16_t xv = (uint16_t)(x[h] >> (16 * half));
                        const uint16_t hv = (uint16_t)(f.kx[i][h] >> (16 * half));
                        const uint16_t lv = (uint16_t)(f.kn[i][h] >> (16 * half));
                        a |= (uint32_t)(bf2f(xv) > bf2f(hv) ? xv : hv) << (16 * half);
                        b |= (uint32_t)(bf2f(xv) < bf2f(lv) ? xv : lv) << (16 * half);
                    }
                    f.kx[i][h] = a;
                    f.kn[i][h] = b;
                }
            }
            const size_t off = ((size_t)u * L.S + p) * D + part * (D / 8) + 8 * i;
            st4((uint16_t*)L.kmax + off, f.kx[i]);
            st4((uint16_t*)L.kmin + off, f.kn[i]);
        }
    }
    const int c0 = part * (D / 8);
    // the keys widened to fp32 once for all heads (exact for bf16)
    float kxf[D / 8], knf[D / 8];
#pragma unroll
    for (int i = 0; i < SV; ++i)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            kxf[8 * i + e] = bf2f(u16_at(f.kx[i], e));
            knf[8 * i + e] = bf2f(u16_at(f.kn[i], e));
        }
    double best = -INFINITY;
#pragma unroll 1
    for (int j = 0; j < G; ++j) {
        const float* qj = qf + (size_t)j * qpad_row(D) + c0 + 4 * part;  // see qpad_index
        double a0 = 0.0, a1 = 0.0;  // even and odd channels
#pragma unroll
        for (int c = 0; c < D / 8; c += 4) {
            const float4 qq = *reinterpret_cast<const float4*>(qj + c);
            a0 += (double)fmaxf(qq.x * kxf[c], qq.x * knf[c]);
            a1 += (double)fmaxf(qq.y * kxf[c + 1], qq.y * knf[c + 1]);
            a0 += (double)fmaxf(qq.z * kxf[c + 2], qq.z * knf[c + 2]);
            a1 += (double)fmaxf(qq.w * kxf[c + 3], qq.w * knf[c + 3]);
        }
        double a = a0 + a1;
        // the eight parts: pairs, then quads, then the two quads (the lanes of
        // a quad hold equal sums by then, so the mirror partner gives lane ^ 4's)
        a += dpp_f64<0xB1>(a);
        a += dpp_f64<0x4E>(a);
        a += dpp_f64<0x141>(a);
        best = a > best ? a : best;
        if (hb != nullptr && part == 0) hb[j] = a;  // per-head bounds, for the softmax aggregation
    }
    return best;
}

// Order-preserving map of a float onto an int (for an LDS atomic minimum), and back.
__device__ __forceinline__ int float_order(float x) {
    const int i = __builtin_bit_cast(int, x);
    return i >= 0 ? i : i ^ 0x7FFFFFFF;
}
__device__ __forceinline__ float order_float(int i) { return __builtin_bit_cast(float, i >= 0 ? i : i ^ 0x7FFFFFFF); }

// Order-preserving unsigned key of a float (unsigned order = numeric order,
// -0 just below +0), and back.
__device__ __forceinline__ unsigned ukey_f32(float x) {
    const unsigned b = __float_as_uint(x);
    return (b >> 31) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float from_ukey_f32(unsigned k) { return __uint_as_float((k >> 31) ? (k & 0x7FFFFFFFu) : ~k); }

// Wavefront 0's part of a pass of a radix select from the top: hist[0 .. 255]
// holds the counts of one digit among the keys still in play; finds the bin
// holding the want-th largest of them (1-based) and the rank within that bin,
// into hist[256] and hist[257]. Lane l scans bins 255-4l .. 252-4l.
__device__ __forceinline__ void radix_pick_top(int* hist, int want, int lane) {
    const int c0 = hist[255 - 4 * lane], c1 = hist[254 - 4 * lane], c2 = hist[253 - 4 * lane],
              c3 = hist[252 - 4 * lane];
    const int sum = c0 + c1 + c2 + c3;
    int incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off);
        if (lane >= off) incl += v;
    }
    const int excl = incl - sum;
    if (excl < want && want <= incl) {
        int r = want - excl, b = 255 - 4 * lane;
        if (r > c0) {
            r -= c0;
            --b;
            if (r > c1) {
                r -= c1;
                --b;
                if (r > c2) {
                    r -= c2;
                    --b;
                }
            }
        }
        hist[256] = b;
        hist[257] = r;
    }
}

// Per bf16 half: the magnitude, at least the smallest normal (2^-126).
__device__ __forceinline__ uint32_t mag_floor(uint32_t x) {
    uint32_t lo = x & 0x7FFFu, hi = (x >> 16) & 0x7FFFu;
    lo = lo < 0x80u ? 0x80u : lo;
    hi = hi < 0x80u ? 0x80u : hi;
    return lo | (hi << 16);
}

// Quest bounds of the pages in slots 0 .. npages-1 (max over the heads of
// sum_c max(q_c kmax_c, q_c kmin_c), Section 4.2 with Quest's page
// representatives), as intervals, on the MFMA. With q+ and q- the positive
// and negative parts of q, a channel's term is q+ kmax + q- kmin, so per
// tile of 16 pages the bounds of every head are the product of [kmax | kmin]
// (pages x 2D) with [q+ ; q-] (2D x heads). The fp32 sum B of those 2D exact
// products lies within 2D 2^-23 E of the exact one whichever way each
// addition rounds, E the sum of their magnitudes; a product flushed for a
// subnormal factor or result loses at most what the same product of
// magnitudes floored at 2^-126 keeps, or 2^-126. So, with E taken over the
// floored magnitudes (one more product on the MFMA), the exact bound lies in
// B -+ (2^-13 E + 1e-30) at D up to 128, with room for E's own rounding.
// Written to lo/hi, with (-inf, inf) where a sum is not finite. Each
// wavefront takes tiles w, w + NW, ..., TPW of them loaded at once. q_ops:
// this lane's query operands (heads as columns). issue: the caller's loads,
// issued behind the last round of tiles on every wavefront.
template <int D, int NW, bool NT, class Issue>
__device__ __forceinline__ void prompt_bounds(const LayerView& L, size_t base, int npages, const bf16x8 (&q_ops)[D / 32],
                                              float* lo, float* hi, Issue&& issue) {
    constexpr int KS = D / 32, TPW = D >= 128 ? 2 : 4;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, grp = lane >> 4, col = lane & 15;
    u32x4 qpos[KS], qneg[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const u32x4 x = __builtin_bit_cast(u32x4, q_ops[ks]);
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const uint32_t neg = ((x[h] >> 15) & 0x00010001u) * 0xFFFFu;  // halves with the sign set
            qneg[ks][h] = x[h] & neg;
            qpos[ks][h] = x[h] & ~neg;
        }
    }
    auto mfma = [](u32x4 a, u32x4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                       0, 0, 0);
    };
    auto floored = [](u32x4 x) { return u32x4{mag_floor(x[0]), mag_floor(x[1]), mag_floor(x[2]), mag_floor(x[3])}; };
    const int ntile = (npages + 15) / 16;
    constexpr int RT = TPW * NW;  // tiles per round of the workgroup
    const int nround = w < ntile ? (ntile - w + RT - 1) / RT : 0;  // rounds of this wavefront
    // lane (grp, col) supplies page 16t + col's channels 32ks + 8grp .. +7
    // (rows past npages, and tiles past the last, repeat the last page and
    // are not written)
    auto load = [&](int t0, u32x4 (&ax)[TPW][KS], u32x4 (&an)[TPW][KS]) {
#pragma unroll
        for (int h = 0; h < TPW; ++h) {
            const int t = min(t0 + h * NW, ntile - 1);
            const size_t off = (base + min(16 * t + col, npages - 1)) * D + 8 * grp;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const uint16_t* px = (const uint16_t*)L.kmax + off + 32 * ks;
                const uint16_t* pn = (const uint16_t*)L.kmin + off + 32 * ks;
                if constexpr (NT) {
                    ax[h][ks] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(px));
                    an[h][ks] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(pn));
                } else {
                    ax[h][ks] = ld4(px);
                    an[h][ks] = ld4(pn);
                }
            }
        }
    };
    auto bound = [&](int t0, const u32x4 (&ax)[TPW][KS], const u32x4 (&an)[TPW][KS]) {
#pragma unroll
        for (int h = 0; h < TPW; ++h) {
            const int t = t0 + h * NW;  // (a tile past the last is computed and not written)
            f32x4 sb = {0.f, 0.f, 0.f, 0.f}, se = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                sb = mfma(ax[h][ks], qpos[ks], sb);
                sb = mfma(an[h][ks], qneg[ks], sb);
                se = mfma(floored(ax[h][ks]), floored(qpos[ks]), se);
                se = mfma(floored(an[h][ks]), floored(qneg[ks]), se);
            }
            // lane (grp, col) holds head col of pages 16t + 4grp + i: the max over the heads
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float bm = col < L.G ? sb[i] : -INFINITY, em = col < L.G ? se[i] : 0.0f;
#pragma unroll
                for (int o = 8; o >= 1; o >>= 1) {
                    bm = fmaxf(bm, __shfl_xor(bm, o));
                    em = fmaxf(em, __shfl_xor(em, o));
                }
                const int p = 16 * t + 4 * grp + i;
                if (col == 0 && p < npages) {
                    const float err = em * 1.220703125e-04f + 1e-30f;  // 2^-13 E + 1e-30
                    const bool fin = __builtin_isfinite(bm) && __builtin_isfinite(err);
                    lo[p] = fin ? bm - err : -INFINITY;
                    hi[p] = fin ? bm + err : INFINITY;
                }
            }
        }
    };
    for (int r = 0; r + 1 < nround; ++r) {
        u32x4 ax[TPW][KS], an[TPW][KS];
        load(w + r * RT, ax, an);
        bound(w + r * RT, ax, an);
    }
    // the last round: its tiles, then the caller's loads, which the wait for
    // the tiles leaves in flight (loads complete in issue order); a wavefront
    // with no tile loads the last one and writes nothing
    const int tl = w + max(nround - 1, 0) * RT;
    u32x4 ax[TPW][KS], an[TPW][KS];
    load(tl, ax, an);
    __builtin_amdgcn_sched_barrier(0);  // (the caller's loads stay behind the tiles')
    issue();
    __builtin_amdgcn_sched_barrier(0);
    bound(tl, ax, an);
}

// Results of the retention policy for one step, computed by the retention
// wavefront and applied to the pool once the attention has read it.
struct RetShared {
    int victim, evicted, next_slot, next_fill, tail_after, errs;
};

// Page scores of the softmax aggregation, by a whole workgroup (every
// thread calls it): for each query head, a softmax over the ranked pages of
// the head's bounds b (scale c = 1/sqrt(D), shifted by the head's largest
// bound M), summed over the heads in head order: score(p) = sum_hj
// exp(c (b_hj(p) - M_hj)) / Z_hj. The heads are the G of each of nu units
// deciding together; hb[((h*S) + p)*G + j] holds head j of unit h's bound of
// page p for every ranked page p. First one wavefront per head finds M and Z
// (into s_mz), then one thread per page sums its terms; s_score is visible
// to the whole workgroup on return.
__device__ void softmax_sum_block(const LayerView& L, const double* hb, int nu, const int* s_state,
                                  double* s_score, double* s_mz, int tid, int nthreads) {
    const int S = L.S, G = L.G, H = nu * G, lane = tid & 63, nw = nthreads >> 6;
    const double c = 1.0 / sqrt((double)L.D);
    for (int hj = tid >> 6; hj < H; hj += nw) {
        const int h = hj / G, j = hj - (hj / G) * G;
        const double* hbj = hb + (size_t)h * S * G + j;
        double mx = -INFINITY;
        for (int p = lane; p < S; p += 64)
            if (ranked(L, s_state[p])) mx = fmax(mx, hbj[(size_t)p * G]);
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mx = fmax(mx, __shfl_xor(mx, off));
        double z = 0.0;
        for (int p = lane; p < S; p += 64)
            if (ranked(L, s_state[p])) z += exp(c * (hbj[(size_t)p * G] - mx));
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) z += __shfl_xor(z, off);
        if (lane == 0) {
            s_mz[2 * hj] = mx;
            s_mz[2 * hj + 1] = z;
        }
    }
    __syncthreads();
    for (int p = tid; p < S; p += nthreads) {
        if (!ranked(L, s_state[p])) continue;
        double acc = 0.0;
#pragma unroll 8
        for (int hj = 0; hj < H; ++hj) {
            const int h = hj / G, j = hj - (hj / G) * G;
            acc += exp(c * (hb[((size_t)h * S + p) * G + j] - s_mz[2 * hj])) / s_mz[2 * hj + 1];
        }
        s_score[p] = acc;
    }
    __syncthreads();
}

// Retention policy of one unit, run by one wavefront (Algorithm 1, the
// decode-stage cache store; Sections 3.2-3.3) on the slot state in LDS, the opened page
// already marked evictable and s_score holding every ranked page's score
// (+inf elsewhere):
//  - top-r refresh: with n ranked pages and k = floor(r*n), an evictable
//    page p gets ts = clock when at least n-k ranked pages score strictly
//    less, i.e. exactly the pages above the (n-k)-th smallest score (the
//    ranked pages are the evictable ones, plus the pinned ones when the pool
//    ranks them; pinned pages never take a timestamp);
//  - eviction (Algorithm 1, the eviction branch of the decode-stage store):
//    when the tail page is full and no slot is free, the evictable page with
//    the smallest (timestamp, logical id) is freed;
//  - the next token's target: the tail page if it has room, else the lowest
//    free slot (a fresh page).
__device__ void evict_wave(const LayerView& L, const UnitRec& ur, int* s_state, int* s_ts, const int* s_lid,
                           RetShared& out);

// lo: where the rank count starts, at most the first slot that a ranked
// page can occupy (slots below the decode base, and below the unit's pinned
// pages unless the pool ranks them, hold none).
__device__ void retention_wave(const LayerView& L, const UnitRec& ur, double r, const double* s_score,
                               int* s_state, int* s_ts, const int* s_lid, RetShared& out, int lo) {
    const int S = L.S, lane = threadIdx.x & 63, s_lo = lo;
    int n = 0;
    for (int s0 = s_lo; s0 < S; s0 += 64) {
        const int s = s0 + lane;
        const int st = s < S ? s_state[s] : -1;
        n += __popcll(__ballot(st >= 0 && ranked(L, st)));
    }
    const int k = (int)floor(r * (double)n);
    if (k > 0) {
        for (int s0 = s_lo; s0 < S; s0 += 64) {
            const int p = s0 + lane;
            if (p < S && s_state[p] == kEvictable) {
                const double sp = s_score[p];
                int less = 0;
#pragma unroll 8
                for (int o = s_lo; o < S; ++o) less += s_score[o] < sp;
                if (less >= n - k) s_ts[p] = ur.clock;
            }
        }
    }
    evict_wave(L, ur, s_state, s_ts, s_lid, out);
}

// Eviction and the next token's target, by one wavefront, once the refresh
// has set the timestamps.
__device__ void evict_wave(const LayerView& L, const UnitRec& ur, int* s_state, int* s_ts, const int* s_lid,
                           RetShared& out) {
    const int S = L.S, ps = L.ps, lane = threadIdx.x & 63;
    int nfree = 0;  // free decode slots
    for (int s0 = L.dbase; s0 < S; s0 += 64) {
        const int s = s0 + lane;
        nfree += __popcll(__ballot(s < S && s_state[s] == kFree));
    }
    const int fill_tail = ur.nf + 1;
    const bool full = fill_tail == ps && nfree == 0;
    int victim = -1;
    if (full) {
        unsigned long long best = ~0ull;
        for (int s0 = L.dbase; s0 < S; s0 += 64) {  // no decode page lies below the decode base
            const int s = s0 + lane;
            if (s < S && s_state[s] == kEvictable) {
                const unsigned long long key = ((unsigned long long)(uint32_t)s_ts[s] << 32) | (uint32_t)s_lid[s];
                best = key < best ? key : best;
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const unsigned long long o = __shfl_xor(best, off);
            best = o < best ? o : best;
        }
        for (int s0 = L.dbase; s0 < S; s0 += 64) {
            const int s = s0 + lane;
            const bool hit = s < S && s_state[s] == kEvictable &&
                             (uint32_t)s_lid[s] == (uint32_t)(best & 0xFFFFFFFFull);
            const unsigned long long m = __ballot(hit);
            if (m) {
                victim = s0 + __builtin_ctzll(m);
                break;
            }
        }
    }
    const bool tail_gone = victim == ur.ns;
    const int tail_fill = tail_gone ? 0 : fill_tail;
    const bool need_free = tail_gone || tail_fill == ps;
    int next_slot = ur.ns;
    if (need_free) {
        next_slot = S;
        for (int s0 = L.dbase; s0 < S; s0 += 64) {
            const int s = s0 + lane;
            const unsigned long long m = __ballot(s < S && (s_state[s] == kFree || s == victim));
            if (m) {
                next_slot = s0 + __builtin_ctzll(m);
                break;
            }
        }
    }
    if (lane == 0) {
        out.victim = victim;
        out.evicted = victim >= 0 ? s_lid[victim] : -1;
        out.next_slot = next_slot < S ? next_slot : 0;
        out.next_fill = need_free ? 0 : tail_fill;
        out.tail_after = tail_gone ? -1 : ur.ns;
        out.errs = (full && victim < 0 ? 2 : 0) | (need_free && next_slot >= S ? 4 : 0);
    }
    if (victim >= 0 && lane == 0) {
        s_state[victim] = kFree;
        s_ts[victim] = -1;
    }
}

// Order-preserving 64-bit key of a finite double (unsigned order = numeric
// order, with -0 just below +0), and back.
__device__ __forceinline__ unsigned long long order_key(double x) {
    const unsigned long long b = (unsigned long long)__double_as_longlong(x);
    return (b >> 63) ? ~b : (b | (1ull << 63));
}
__device__ __forceinline__ double from_order_key(unsigned long long k) {
    return __longlong_as_double((long long)((k >> 63) ? (k & ~(1ull << 63)) : ~k));
}

// kth_largest_wg for doubles: eight 8-bit digits of order_key (-0 counted as
// +0, which it equals), by a workgroup of nth threads. hist: 258 ints.
__device__ double kth_largest_f64_wg(const double* x, int n, int k, int* hist, int tid, int nth) {
    const int lane = tid & 63;
    unsigned long long prefix = 0;
    int want = k;
    for (int shift = 56; shift >= 0; shift -= 8) {
        for (int b = tid; b < 256; b += nth) hist[b] = 0;
        __syncthreads();
        const unsigned long long high = shift == 56 ? 0ull : ~0ull << (shift + 8);
        for (int p = tid; p < n; p += nth) {
            const unsigned long long key = order_key(x[p] + 0.0);
            if ((key & high) == prefix) atomicAdd(&hist[(int)((key >> shift) & 255ull)], 1);
        }
        __syncthreads();
        if (tid < 64) radix_pick_top(hist, want, lane);
        __syncthreads();
        prefix |= (unsigned long long)hist[256] << shift;
        want = hist[257];
    }
    return from_order_key(prefix);
}

// Top-r refresh by a whole workgroup (every thread calls it; the epilogue
// kernel's version of the rule in retention_wave). With n ranked pages and
// k = floor(r*n), an evictable page is refreshed when at least n-k ranked
// pages score strictly less. Up to 256 slots this is counted directly.
// Beyond, the workgroup finds theta, the (n-k)-th smallest ranked score, by
// a radix select over order_key (eight 8-bit digits, most significant
// first, a 256-bin histogram each) and refreshes the evictable pages
// scoring above theta: the same pages, since fewer than n-k ranked scores
// lie below theta and at least n-k lie at or below it. Slots below first
// hold no ranked page (the prompt region's, when there is one). s_aux: 260
// ints.
__device__ void refresh_block(const LayerView& L, const UnitRec& ur, double r, const double* s_score,
                              const int* s_state, int* s_ts, int* s_aux, int tid, int nthreads, int first) {
    const int S = L.S, lane = tid & 63;
    int* s_hist = s_aux;  // [256]
    if (tid == 0) s_aux[256] = 0;
    __syncthreads();
    int cnt = 0;
    for (int p = first + tid; p < S; p += nthreads) cnt += ranked(L, s_state[p]) ? 1 : 0;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) cnt += __shfl_xor(cnt, off);
    if (lane == 0 && cnt) atomicAdd(&s_aux[256], cnt);
    __syncthreads();
    const int n = s_aux[256];
    const int k = (int)floor(r * (double)n);
    if (k == 0) return;
    if (k == n) {  // every page refreshed
        for (int p = first + tid; p < S; p += nthreads)
            if (s_state[p] == kEvictable) s_ts[p] = ur.clock;
        return;
    }
    if (S - first <= 256) {
        for (int p = first + tid; p < S; p += nthreads) {
            if (s_state[p] != kEvictable) continue;
            const double sp = s_score[p];
            int less = 0;
#pragma unroll 8
            for (int o = first; o < S; ++o) less += s_score[o] < sp;  // unranked slots hold +inf
            if (less >= n - k) s_ts[p] = ur.clock;
        }
        return;
    }
    unsigned long long prefix = 0;
    int want = n - k - 1;  // 0-based rank of theta among the ranked scores
    for (int shift = 56; shift >= 0; shift -= 8) {
        for (int b = tid; b < 256; b += nthreads) s_hist[b] = 0;
        __syncthreads();
        const unsigned long long high = shift == 56 ? 0ull : (~0ull << (shift + 8));
        for (int p = first + tid; p < S; p += nthreads) {
            if (!ranked(L, s_state[p])) continue;
            const unsigned long long key = order_key(s_score[p]);
            if ((key & high) == prefix) atomicAdd(&s_hist[(int)((key >> shift) & 255ull)], 1);
        }
        __syncthreads();
        if (tid < 64) {  // wavefront 0 scans the bins: lane l holds bins 4l .. 4l+3
            const int c0 = s_hist[4 * lane], c1 = s_hist[4 * lane + 1], c2 = s_hist[4 * lane + 2],
                      c3 = s_hist[4 * lane + 3];
            const int sum = c0 + c1 + c2 + c3;
            int incl = sum;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int v = __shfl_up(incl, off);
                if (lane >= off) incl += v;
            }
            const int excl = incl - sum;
            if (excl <= want && want < incl) {
                int w = want - excl, b = 4 * lane;
                if (w >= c0) {
                    w -= c0;
                    ++b;
                    if (w >= c1) {
                        w -= c1;
                        ++b;
                        if (w >= c2) {
                            w -= c2;
                            ++b;
                        }
                    }
                }
                s_aux[257] = b;
                s_aux[258] = w;
            }
        }
        __syncthreads();
        prefix |= (unsigned long long)s_aux[257] << shift;
        want = s_aux[258];
    }
    const double theta = from_order_key(prefix);
    for (int p = first + tid; p < S; p += nthreads)
        if (s_state[p] == kEvictable && s_score[p] > theta) s_ts[p] = ur.clock;
}

// Writes the step's retention results to the pool and the optional outputs.
__device__ void retention_store(const LayerView& L, const StepIO& io, int u, const UnitRec& ur,
                                const int* s_state, const int* s_ts, const int* s_lid, const RetShared& rs,
                                int first, int stride) {
    const int S = L.S;
    const size_t base = (size_t)u * S;
    for (int s = first; s < S; s += stride) {
        const bool gone = s == rs.victim;
        const int st = s_state[s];
        const int id = gone ? -1 : s_lid[s];
        if (st == kEvictable || gone) L.ts[base + s] = s_ts[s];
        if (s == ur.ns || gone) {
            L.state[base + s] = st;
            L.lid[base + s] = id;
            L.fill[base + s] = gone ? 0 : ur.nf + 1;
        }
        if (io.page_table_out) io.page_table_out[base + s] = (st == kFree) ? -1 : id;
        if (io.timestamps_out) io.timestamps_out[base + s] = (st == kEvictable) ? s_ts[s] : -1;
    }
    if (first == 0) {
        int32_t* U4 = L.unit + (size_t)u * kUnitFields;
        U4[kTail] = rs.tail_after;
        U4[kNextLid] = ur.next_lid + (ur.opened() ? 1 : 0);
        U4[kClock] = ur.clock + 1;
        U4[kEvicted] = rs.evicted;
        U4[kNextSlot] = rs.next_slot;
        U4[kNextFill] = rs.next_fill;
        if (io.evicted_out) io.evicted_out[u] = rs.evicted;
        if (rs.errs) atomicOr(L.err, rs.errs);
    }
}

// Makes this wavefront's LDS writes visible to its own later LDS reads (the
// lanes of one wavefront exchanging data through LDS; no workgroup barrier).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waits for every vector-memory load in flight (vmcnt(0); expcnt and lgkmcnt left at their maxima).
__device__ __forceinline__ void vm_drain() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Workgroup barrier that waits for this wavefront's LDS traffic only: loads
// already issued to global memory stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt left at their maxima
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// The k-th largest of x[0 .. n-1] (1 <= k <= n, counted with multiplicity),
// by a whole workgroup of NT threads (every thread calls it and gets the
// value): a radix select over ukey_f32, four 8-bit digits from the most
// significant, a 256-bin histogram of the keys that match the digits found
// so far in each pass; wavefront 0 scans the bins from the top for the one
// holding the k-th key. hist: 258 ints of LDS.
template <int NT>
__device__ float kth_largest_wg(const float* x, int n, int k, int* hist, int tid) {
    const int lane = tid & 63;
    unsigned prefix = 0;
    int want = k;  // rank from the top among the keys that match prefix, 1-based
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int b = tid; b < 256; b += NT) hist[b] = 0;
        lds_barrier();
        const unsigned high = shift == 24 ? 0u : ~0u << (shift + 8);
        for (int p = tid; p < n; p += NT) {
            const unsigned key = ukey_f32(x[p]);
            if ((key & high) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
        }
        lds_barrier();
        if (tid < 64) radix_pick_top(hist, want, lane);
        lds_barrier();
        prefix |= (unsigned)hist[256] << shift;
        want = hist[257];
    }
    return from_ukey_f32(prefix);
}

// One 32-token block of attention for the GQA group held by this wavefront:
// QK^T as two 16x16x32 bf16 MFMA tiles per 32 channels (rows = tokens,
// columns = query heads), online softmax in base 2 with one cross-lane max,
// PV as D/16 MFMAs of V^T times P^T. nv: valid rows among this lane's eight.
template <int D>
__device__ __forceinline__ void attend_block(const u32x4 (&kr)[2][D / 32], const u32x4 (&vr)[D / 16], int nv,
                                             const bf16x8 (&qv)[D / 32], float scale_log2, float& m_run,
                                             float& l_run, f32x4 (&acc)[D / 16]) {
    constexpr int KS = D / 32, NB = D / 16;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[0][ks]), qv[ks], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kr[1][ks]), qv[ks], s1, 0, 0, 0);
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
    mb = max_xor16_32(mb);
    const float m_new = fmaxf(m_run, mb);
    if (__ballot(m_new > m_run) != 0ull) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb] *= alpha;
        m_run = m_new;
    }
    float psum = 0.0f;
    bf16x8 pb;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float pj = __builtin_amdgcn_exp2f(x[j] - m_run);
        psum += pj;
        pb[j] = (__bf16)pj;
    }
    l_run += psum;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vr[nb]), pb, acc[nb], 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Step kernel, bf16 pools. One workgroup of NW wavefronts per (unit, split).
//
// Attention (Algorithm 1, attention(Q, K_old::K_new, V_old::V_new)) over
// every resident token, split-K over 32-token blocks. Each wavefront holds
// the unit's whole GQA query group; it takes one block statically, then
// claims further blocks from a counter in LDS, so the wavefronts that the
// memory system serves faster take more blocks. The next block loads while
// the current one computes. Per block: QK^T as two 16x16x32 bf16 MFMA tiles
// per 32 channels (rows = tokens, columns = query heads, G <= 16 of the 16
// used), online softmax in base 2 with one cross-lane max per block, and PV
// as D/16 MFMAs of V^T (rows = channels) times P^T (columns = heads). A lane
// owns one head (its column) in both products, so no data moves between
// lanes except the block max. The new token is not in the pool when the
// block is read: its K/V come from the step's inputs, substituted in
// registers, and the wavefront holding that block stores it.
//
// Page-score passes ride along with the first blocks. Once every wavefront
// has finished its passes (a workgroup barrier), wavefront 0 runs the
// retention policy when one workgroup covers the unit (fused), then goes on
// claiming blocks. The state reaches the pool only after the attention has
// read it; the wavefronts' partial outputs merge at the end, into the output
// when one workgroup covers the unit, else into the split's partial.

// AGG: the softmax aggregation of the page scores (a separate instance, so
// that the default one carries none of its registers).
// LM, pools with a prompt region (Quest on the prompt): 1, the blocks come
// from the unit's block list (the prompt blocks the selection kernel chose,
// then the decode region's); 2, the workgroup covers the unit and selects the
// prompt pages itself before its block loop (bounds on the MFMA, exact ones
// for the pages near the cut), then claims the decode blocks and the chosen
// prompt blocks from one list. 0: no prompt region.
// NT: K/V blocks are read with non-temporal loads (pools too large for the
// memory-side cache to serve the next step).
// The step of work item wi = unit * nsplit + split, by one workgroup (the
// arguments by value: as kernel arguments, they leave the registers of the
// block loop alone).
template <int D, int NW, bool AGG, int LM, bool NT>
__device__ __forceinline__ void step_item(LayerView L, StepIO io, float scale_log2, double r, int fused,
                                          const int wi) {
    constexpr int KS = D / 32, NB = D / 16, BLK = 32 * D;
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ float s_m[NW][16];
    __shared__ float s_l[NW][16];
    __shared__ RetShared ret;
    __shared__ int s_next;  // next unclaimed block index
    __shared__ int s_nsel;  // LM 2: prompt blocks chosen
    __shared__ int s_lo;    // LM 2: the topk-th largest lower end of a prompt bound (ordered bits)
    __shared__ int s_ncand; // LM 2: candidate prompt pages
    __shared__ __align__(16) uint16_t s_kn[D];  // the new token's key and value, staged so that
    __shared__ __align__(16) uint16_t s_vn[D];  // no read in the block loop waits on memory

    const int G = L.G, S = L.S, ps = L.ps;
    float* s_qf = reinterpret_cast<float*>(smem);  // [G][D+32] q in fp32, padded: qpad_index
    float* s_o = s_qf + (size_t)G * qpad_row(D);   // [NW][G][D+4]
    double* s_score = reinterpret_cast<double*>(s_o + (size_t)NW * G * (D + 4));  // [S], fused only
    double* s_hb = s_score + S;  // [S][G] per-head bounds, fused softmax aggregation only
    double* s_mz = s_hb + (AGG ? (size_t)S * G : 0);  // [G][2] each head's M and Z, likewise
    int* s_state = reinterpret_cast<int*>(s_mz + (AGG ? 2 * G : 0));  // [S], fused only
    int* s_ts = s_state + S;
    int* s_lid = s_ts + S;
    int* s_list = fused ? s_lid + S : reinterpret_cast<int*>(s_score);  // LM 1: this workgroup's blocks
    // LM 2: the prompt pages' bound intervals and attended fills, the chosen
    // prompt blocks, the candidate pages and their exact bounds
    float* s_plo = reinterpret_cast<float*>(  // [dbase] lower ends, 16-byte aligned (the smem base is)
        reinterpret_cast<int*>(smem) + ((s_lid + S - reinterpret_cast<int*>(smem) + 3) & ~3));
    float* s_phi = s_plo + L.dbase;                                // [dbase] upper ends
    int* s_fatt = reinterpret_cast<int*>(s_phi + L.dbase);         // [dbase]
    int* s_plist = s_fatt + L.dbase;                               // [dbase * ps / 32]
    int* s_cand = s_plist + L.dbase * ps / 32;                     // [dbase]
    double* s_ex = reinterpret_cast<double*>(                      // [dbase], 8-byte aligned
        reinterpret_cast<int*>(smem) + ((s_cand + L.dbase - reinterpret_cast<int*>(smem) + 1) & ~1));

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 4, col = lane & 15;
    const int nsplit = L.nsplit;
    const unsigned uwi = (unsigned)wi;  // (unsigned arithmetic, as on blockIdx.x)
    const int u = uwi / nsplit, split = uwi - (uwi / nsplit) * nsplit;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;  // the sequence sits this step out
    const size_t base = (size_t)u * S;
    // this workgroup's claims lo .. hi-1: blocks of the unit (a range), or
    // (LIST) entries of its block list; pages scored here: those whose first
    // row lies in blocks sb0 .. sb1-1
    int lo, hi, sb0, sb1;
    const int nbp = LM ? L.dbase * ps / 32 : 0;  // LM: the decode region starts at this block
    if constexpr (LM == 2) {
        lo = 0;
        hi = L.nblk - nbp;  // decode blocks, claimed first; claims beyond are the chosen prompt blocks
        sb0 = nbp;          // score passes: the decode pages
        sb1 = L.nblk;
    } else if constexpr (LM == 1) {
        const int nsel = L.bcnt[2 * u], ntot = L.bcnt[2 * u + 1];
        const int per = (ntot + nsplit - 1) / nsplit;
        lo = min(ntot, split * per);
        hi = min(ntot, lo + per);
        sb0 = nbp + max(lo, nsel) - nsel;
        sb1 = nbp + max(hi, nsel) - nsel;
        for (int i = tid; i < hi - lo; i += NW * 64) s_list[i] = L.blist[(size_t)u * L.lcap_blk + lo + i];
        __syncthreads();
    } else {
        lo = split * L.bps;
        hi = max(lo, min(L.nblk, lo + L.bps));
        sb0 = lo;
        sb1 = hi;
    }
    const int nown = hi - lo;                  // claims of this workgroup
    const int bend = LM ? 0x40000000 : hi;     // no block: every block index lies below
    auto real = [&](int x) { return x < bend; };
    const uint16_t* qg = (const uint16_t*)io.q + (size_t)u * G * D;
    const uint16_t* kn_g = (const uint16_t*)io.k_new + (size_t)u * D;
    const uint16_t* vn_g = (const uint16_t*)io.v_new + (size_t)u * D;
    const uint16_t* Ku = (const uint16_t*)L.K + (size_t)u * L.Lcap * D;
    const uint16_t* Vu = (const uint16_t*)L.V + (size_t)u * L.Lcap * D;
    // fills the attention sees (the plain fill pointer where they are the
    // same: read through it, the first block's fill arrives sooner)
    const int32_t* fu = (LM == 1 ? L.fill_att : L.fill) + base;
    auto ldb = [&](const uint16_t* p) {
        if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        else return ld4(p);
    };
    auto load_block = [&](int b, u32x4 (&kr)[2][KS], u32x4 (&vr)[NB]) {
        const uint16_t* Kb = Ku + (size_t)b * BLK + lane * 8;
        const uint16_t* Vb = Vu + (size_t)b * BLK + lane * 8;
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kr[qq][ks] = ldb(Kb + (qq * KS + ks) * 512);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) vr[nb] = ldb(Vb + nb * 512);
    };

    // Loads complete in issue order, so the small reads go out first: the
    // unit record, this thread's staging elements and slot, the first
    // block's fill and the queries; then the first block (its index w is
    // static), which the staging below no longer waits for (LM 2: the
    // staging, then the bound tiles, then the first block).
    const int32_t* U4 = L.unit + (size_t)u * kUnitFields;
    const UnitRec ur{U4[kNextSlot], U4[kNextFill], U4[kClock], U4[kNextLid]};
    const int pinned = U4[kPinnedPages];
    // claim index i of the own blocks, ascending or (L.rev) descending
    auto blk_of = [&](int i) {
        const int j = L.rev ? nown - 1 - i : i;
        if constexpr (LM == 1) return s_list[j];
        else if constexpr (LM == 2) return nbp + j;
        else return lo + j;
    };
    int b = (w < nown) ? blk_of(w) : bend;  // (LM 2: a prompt block, once they are chosen)
    const int slot_first = (32 * b + 8 * grp) / ps;
    const int fill_first = (real(b) && slot_first < S) ? fu[slot_first] : 0;
    // unconditional (clamped) reads: a read under a branch draws its first
    // use into the branch, with a wait for it ahead of the block loads
    const uint16_t q_first = qg[tid < G * D ? tid : 0];
    const int t_new = tid < D / 8 ? tid : 0;
    const u32x4 kn_first = ld4(kn_g + 8 * t_new), vn_first = ld4(vn_g + 8 * t_new);
    const int s_first = tid < S ? tid : 0;
    const int st_first = L.state[base + s_first], ts_first = L.ts[base + s_first], lid_first = L.lid[base + s_first];
    const int pf_first = LM == 2 ? fu[tid < L.dbase ? tid : 0] : 0;  // LM 2: a prompt page's fill
    // LM 2: a second slot and prompt page per thread, with the reads above
    const int sl_sec = tid + NW * 64 < S ? tid + NW * 64 : 0, pg_sec = tid + NW * 64 < L.dbase ? tid + NW * 64 : 0;
    int st_sec = 0, ts_sec = 0, lid_sec = 0, pf_sec = 0;
    if constexpr (LM == 2) {
        st_sec = L.state[base + sl_sec];
        ts_sec = L.ts[base + sl_sec];
        lid_sec = L.lid[base + sl_sec];
        pf_sec = fu[pg_sec];
    }
    bf16x8 qv[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const u32x4 x = (col < G) ? ld4(qg + (size_t)col * D + 32 * ks + 8 * grp) : u32x4{0u, 0u, 0u, 0u};
        qv[ks] = __builtin_bit_cast(bf16x8, x);
    }
    u32x4 kr_next[2][KS], vr_next[NB];
    int f_first = 0;  // LM 2: the first block's fill
    if constexpr (LM == 2) {
        // The staging first (the other instances stage below, behind the first
        // block's loads), so that none of its reads waits behind the bound
        // tiles or the block: they go out about when the tiles would, which
        // wait for the queries anyway.
        if (tid < L.dbase) s_fatt[tid] = tid < pinned ? pf_first : 0;  // the kept prompt pages' fills
        if (tid + NW * 64 < L.dbase) s_fatt[tid + NW * 64] = tid + NW * 64 < pinned ? pf_sec : 0;
        for (int p = tid + 2 * NW * 64; p < L.dbase; p += NW * 64) s_fatt[p] = p < pinned ? fu[p] : 0;
        // q in fp32 from the query operands: lane (grp, col < G) holds head
        // col's channels 32 ks + 8 grp .. +7, one padded row segment; the
        // wavefronts take turns over ks
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks % NW == w && col < G) {
                const u32x4 x = __builtin_bit_cast(u32x4, qv[ks]);
                float* d = s_qf + qpad_index<D>(col * D + 32 * ks + 8 * grp);
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    d[2 * h] = __uint_as_float(x[h] << 16);
                    d[2 * h + 1] = __uint_as_float(x[h] & 0xFFFF0000u);
                }
            }
        }
        if (tid < D / 8) {
            st4(&s_kn[8 * tid], kn_first);
            st4(&s_vn[8 * tid], vn_first);
        }
        if (fused) {  // (always, with LM 2)
            if (tid < S) stage_slot(ur, tid, st_first, ts_first, lid_first, s_score, s_state, s_ts, s_lid);
            if (tid + NW * 64 < S) stage_slot(ur, tid + NW * 64, st_sec, ts_sec, lid_sec, s_score, s_state, s_ts, s_lid);
            load_slots(L, u, ur, s_score, s_state, s_ts, s_lid, 2 * NW * 64);
        }
        if (tid == 0) {
            s_next = 2 * NW;  // claims start after the two static blocks of every wavefront
            s_lo = 0x7FFFFFFF;
            s_ncand = 0;
        }
        if (w < nown) f_first = slot_first < S ? (slot_first == ur.ns ? ur.nf + 1 : fill_first) : 0;
        // nothing else is in flight yet: every read has landed from here on,
        // also to the compiler, which loses count of loads issued in loops
        vm_drain();
        // the prompt region's bound intervals (the selection reads those of the
        // kept pages), and behind their last loads the first block, which
        // streams during the selection; a wavefront with no decode block reads
        // block 0 and drops it (loads on every path keep the waits for the
        // tiles short of the block)
        auto first = [&]() { load_block(real(b) ? b : 0, kr_next, vr_next); };
        if (L.dbase > L.topk) prompt_bounds<D, NW, NT>(L, base, L.dbase, qv, s_plo, s_phi, first);
        else first();
    } else {
        if (real(b)) load_block(b, kr_next, vr_next);
    }

    const int ns = ur.ns, nf = ur.nf;
    const bool opened = ur.opened();
    const int row_new = ns * ps + nf, b_new = row_new >> 5, tt_new = row_new & 31;
    bool decided = false;  // this wavefront has passed the score barrier
    // the block of claim index i, or bend when none is left (LM 2: the decode
    // blocks, then the chosen prompt blocks)
    auto take = [&](int i) {
        if constexpr (LM == 2) {
            if (i < nown) return blk_of(i);
            return i - nown < s_nsel ? s_plist[i - nown] : bend;
        } else {
            return i < nown ? blk_of(i) : bend;
        }
    };
    // pages scored here: those whose first row lies in this workgroup's blocks, pinned ones
    // excepted unless they are ranked
    const int sl0 = max(L.rank_pinned ? 0 : pinned, min(S, (32 * sb0 + ps - 1) / ps));
    const int sl1 = min(S, (32 * sb1 + ps - 1) / ps);

    // fill of the page holding this lane's 8 rows of block b (page_size % 8 == 0)
    auto row_fill = [&](int b) {
        const int slot = (32 * b + 8 * grp) / ps;
        if constexpr (LM == 2)
            if (slot < L.dbase) return s_fatt[slot];  // read only once the prompt pages are chosen
        return (slot < S) ? (slot == ns ? nf + 1 : fu[slot]) : 0;
    };
    auto valid_rows = [&](int b, int f) {
        const int t0 = 32 * b + 8 * grp;
        return min(max(f - (t0 - (t0 / ps) * ps), 0), 8);
    };
    int f_next = f_first;
    if constexpr (LM != 2) {
        if (real(b)) f_next = (w < nown) ? (slot_first < S ? (slot_first == ns ? nf + 1 : fill_first) : 0) : row_fill(b);

        // staging for the scores and the epilogue
        if (tid < G * D) s_qf[qpad_index<D>(tid)] = bf2f(q_first);
        for (int i = tid + NW * 64; i < G * D; i += NW * 64) s_qf[qpad_index<D>(i)] = bf2f(qg[i]);
        if (tid < D / 8) {
            st4(&s_kn[8 * tid], kn_first);
            st4(&s_vn[8 * tid], vn_first);
        }
        if (fused) {
            if (tid < S) stage_slot(ur, tid, st_first, ts_first, lid_first, s_score, s_state, s_ts, s_lid);
            load_slots(L, u, ur, s_score, s_state, s_ts, s_lid, NW * 64);
        }
        if (tid == 0) s_next = 2 * NW;  // claims start after the two static blocks of every wavefront
    }
    // the staging is visible: the first block is still in flight, and every
    // wavefront reaches this point after the same short reads
    lds_barrier();

    if constexpr (LM == 2) {
        // the topk kept prompt pages of largest bound, ties to the lower slot
        // (Quest on the prompt): the others' fills are cleared. Each page's
        // exact bound lies in [s_plo, s_phi]; with lo the topk-th largest lower
        // end, at least topk pages have bounds >= lo, so a page whose upper end
        // is below lo ranks below all of them: the top k are among the
        // candidates with upper end >= lo, and rank among them as among all
        // kept pages.
        if (pinned > L.topk && L.topk > 0) {
            float lo_cut;
            if (pinned > 2 * NW * 64) {
                // many kept pages: lo by a radix select (the count below is
                // quadratic in them); s_ex is free until the candidates' bounds
                lo_cut = kth_largest_wg<NW * 64>(s_plo, pinned, L.topk, reinterpret_cast<int*>(s_ex), tid);
            } else {
                const int pin4 = pinned & ~3;
                for (int p = tid; p < pinned; p += NW * 64) {
                    // lower ends above p's: four per 16-byte read, then the last few
                    const float lp = s_plo[p];
                    int above = 0;
#pragma unroll 4
                    for (int o = 0; o < pin4; o += 4) {
                        const float4 x = *reinterpret_cast<const float4*>(s_plo + o);
                        above += (x.x > lp ? 1 : 0) + (x.y > lp ? 1 : 0) + (x.z > lp ? 1 : 0) + (x.w > lp ? 1 : 0);
                    }
                    for (int o = pin4; o < pinned; ++o) above += s_plo[o] > lp ? 1 : 0;
                    if (above < L.topk) atomicMin(&s_lo, float_order(lp));
                }
                lds_barrier();
                lo_cut = order_float(s_lo);
            }
            for (int p = tid; p < pinned; p += NW * 64) {
                if (s_phi[p] >= lo_cut) s_cand[atomicAdd(&s_ncand, 1)] = p;
                else s_fatt[p] = 0;
            }
            lds_barrier();
            // exactly topk candidates: they are the top k; more: the candidates'
            // bounds in fp64, eight lanes per page as the decode pages' scores
            const int nc = s_ncand;
            if (nc > L.topk) {
                for (int c0 = 8 * w; c0 < nc; c0 += 8 * NW) {
                    const int c = c0 + (lane >> 3);
                    const bool act = c < nc;
                    const int p = act ? s_cand[c] : 0;
                    ScoreFrag<D> f;
                    score_issue<D>(L, u, p, lane & 7, act, f);
                    const double sc = score_finish<D>(L, u, p, lane & 7, act, f, false, false, s_kn, s_qf, nullptr);
                    if (act && (lane & 7) == 0) s_ex[c] = sc;
                }
                lds_barrier();
                for (int c = tid; c < nc; c += NW * 64) {
                    const int p = s_cand[c];
                    const double e = s_ex[c];
                    int above = 0;
                    for (int o = 0; o < nc; ++o) {
                        const double x = s_ex[o];
                        above += (x > e || (x == e && s_cand[o] < p)) ? 1 : 0;
                    }
                    if (above >= L.topk) s_fatt[p] = 0;
                }
            }
        }
        lds_barrier();
        if (w == 0) {  // the prompt blocks holding a chosen page, ascending
            int cnt = 0;
            for (int c0 = 0; c0 < nbp; c0 += 64) {
                const int bb = c0 + lane;
                bool any = false;
                if (bb < nbp)
                    for (int sl = 32 * bb / ps; sl <= (32 * bb + 31) / ps; ++sl) any = any || s_fatt[sl] > 0;
                const unsigned long long m = __ballot(any);
                if (any) s_plist[cnt + __popcll(m & ((1ull << lane) - 1ull))] = bb;
                cnt += __popcll(m);
            }
            if (lane == 0) s_nsel = cnt;
        }
        lds_barrier();
        if (w >= nown) {  // no decode block for this wavefront: its first claim is a prompt block
            b = take(w);
            if (b < bend) {
                f_next = row_fill(b);
                load_block(b, kr_next, vr_next);
            }
        }
    }

    float m_run = -INFINITY, l_run = 0.0f;
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    // score passes of this wavefront: 8 pages each, page = first + (lane >> 3)
    const int part = lane & 7;
    const int ngroups = (sl1 - sl0 + 7) / 8;  // 8-page groups, in the step's direction
    auto pass_page = [&](int pass) {
        const int g = pass * NW + w;
        return sl0 + 8 * (L.rev ? ngroups - 1 - g : g) + (lane >> 3);
    };
    auto pass_act = [&](int p) { return p < sl1 && (p == ns || ranked(L, L.state[base + p])); };
    const int npass = (sl1 - sl0 - 8 * w > 0) ? (sl1 - sl0 - 8 * w + 8 * NW - 1) / (8 * NW) : 0;
    const int npass_all = (sl1 - sl0 + 8 * NW - 1) / (8 * NW);  // passes of wavefront 0, the most
    int pass = 0;
    ScoreFrag<D> frag;
    bool act_cur = false;
    auto score_step = [&]() {
        const int p = pass_page(pass);
        double* hb = (AGG && act_cur) ? (fused ? s_hb : L.score + base * G) + (size_t)p * G : nullptr;
        const double sc = score_finish<D>(L, u, p, part, act_cur, frag, p == ns, opened, s_kn, s_qf, hb);
        if (act_cur && part == 0 && !AGG) {
            if (fused) s_score[p] = sc;
            else L.score[base + p] = sc;
        }
        ++pass;
        if (pass < npass) {
            const int pn = pass_page(pass);
            act_cur = pass_act(pn);
            score_issue<D>(L, u, pn, part, act_cur && !(pn == ns && opened), frag);
        }
    };
    // retention policy once every wavefront's scores are in LDS
    auto scores_done = [&]() {
        lds_barrier();
        if (AGG && fused) softmax_sum_block(L, s_hb, 1, s_state, s_score, s_mz, tid, NW * 64);
        // (after the block loop, as with the softmax aggregation, the retention
        // is on the critical path: its count skips the pinned pages; mid-loop
        // it overlaps the streaming, and the narrower count measured no faster)
        if (fused && w == 0)
            retention_wave(L, ur, r, s_score, s_state, s_ts, s_lid, ret,
                           AGG && !L.rank_pinned ? max(L.dbase, pinned) : L.dbase);
        decided = true;
    };

    // after the first block: the first pass's keys start loading
    auto staged = [&]() {
        if (npass > 0) {
            const int p = pass_page(0);
            act_cur = pass_act(p);
            score_issue<D>(L, u, p, part, act_cur && !(p == ns && opened), frag);
        }
    };
    // the first score pass's loads go out now, behind the first blocks' (L.early),
    // or once the first block has been attended and its registers are free
    const int early = L.early;
    if (early) staged();
    int it = 0;
    while (b < bend) {
        const int f_cur = f_next;
        u32x4 kr[2][KS], vr[NB];
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kr[qq][ks] = kr_next[qq][ks];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) vr[nb] = vr_next[nb];
        // one claim per wavefront: from the LDS counter, or (L.det) a fixed
        // interleave, whose partial sums are reproducible
        int bn = bend;
        if (lane == 0) bn = take(L.det ? w + (it + 1) * NW : (it == 0 ? w + NW : atomicAdd(&s_next, 1)));
        bn = __builtin_amdgcn_readfirstlane(bn);
        if (bn < bend) {
            f_next = row_fill(bn);
            load_block(bn, kr_next, vr_next);
        }
        const int nv = valid_rows(b, f_cur);
        if (__ballot(nv > 0) != 0ull) {
            if (b == b_new) {  // the new token: K/V from the inputs
                const int i_new = 4 * (tt_new >> 3) + (tt_new & 3), q_new = (tt_new >> 2) & 1;
                if (col == i_new) {
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) {
                        const u32x4 x = ld4(&s_kn[32 * ks + 8 * grp]);
                        if (q_new == 0) kr[0][ks] = x; else kr[1][ks] = x;
                    }
                }
                if (grp == (tt_new >> 3)) {
                    const int j_new = tt_new & 7;
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb) {
                        const uint32_t val = s_vn[16 * nb + col];
#pragma unroll
                        for (int h = 0; h < 4; ++h) {
                            if ((j_new >> 1) == h) {
                                const int sh = (j_new & 1) * 16;
                                vr[nb][h] = (vr[nb][h] & ~(0xFFFFu << sh)) | (val << sh);
                            }
                        }
                    }
                }
                // append: the new token joins the pool (Algorithm 1, decode-stage store)
                uint16_t* Kw = (uint16_t*)L.K + (size_t)u * L.Lcap * D;
                uint16_t* Vw = (uint16_t*)L.V + (size_t)u * L.Lcap * D;
                if (lane < D / 8) st4(Kw + k_off<D>(row_new, lane * 8), ld4(&s_kn[lane * 8]));
                for (int c = lane; c < D; c += 64) Vw[v_off<D>(row_new, c)] = s_vn[c];
            }

            attend_block<D>(kr, vr, nv, qv, scale_log2, m_run, l_run, acc);
        }
        // this block's registers are free again
        if (it == 0 && !early) {
            staged();
        } else if (pass < npass) {
            score_step();
        }
        // (the softmax aggregation waits for the end of the loop: mid-loop, its
        // arithmetic would compete with the prefetched block for registers;
        // wavefront 0, which has the most passes, has finished them here)
        if (!AGG && it == npass_all - early) scores_done();
        ++it;
        b = bn;
    }
    if (it == 0 && !early) staged();
    while (pass < npass) score_step();  // passes left when the wavefront ran out of blocks
    if (!decided) scores_done();

    // park this wavefront's partial attention in LDS
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
    if (grp == 0) {
        s_m[w][col] = m_run;
        s_l[w][col] = l_run;
    }
    if (col < G) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            *reinterpret_cast<f32x4*>(&s_o[((size_t)w * G + col) * (D + 4) + 16 * nb + 4 * grp]) = acc[nb];
    }
    lds_barrier();  // partials parked, retention decided
    // the state goes out first (every block has been read), its stores
    // draining while the partials merge
    if (fused) retention_store(L, io, u, ur, s_state, s_ts, s_lid, ret, tid, NW * 64);

    // merge the wavefronts' partial outputs
    for (int idx = tid; idx < G * D; idx += NW * 64) {
        const int h = idx / D, c = idx - (idx / D) * D;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) M = fmaxf(M, s_m[ww][h]);
        float O = 0.0f, Ls = 0.0f;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
            const float mw = s_m[ww][h];
            const float wt = (mw == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mw - M);
            O += wt * s_o[((size_t)ww * G + h) * (D + 4) + c];
            Ls += wt * s_l[ww][h];
        }
        if (nsplit == 1) {  // the whole unit: the output itself
            ((uint16_t*)io.out)[((size_t)u * G + h) * D + c] = f2bf(O / Ls);
        } else {
            float* pp = L.part + (((size_t)u * nsplit + split) * G + h) * (D + 2);
            pp[c] = O;
            if (c == 0) {
                pp[D] = M;
                pp[D + 1] = Ls;
            }
        }
    }
}

// Step kernel (bf16 pools): rows a1-a6 for work item blockIdx.x.
template <int D, int NW, bool AGG, int LM, bool NT = false>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_step_bf16(
    LayerView L, StepIO io, float scale_log2, double r, int fused) {
    step_item<D, NW, AGG, LM, NT>(L, io, scale_log2, r, fused, blockIdx.x);
}

// fp32 pools: the step of one split of a unit's rows by one wavefront, over
// its rows in chunks of 64 tokens. In a chunk each lane takes one token: its
// row of K is loaded whole (the loads go out with the unit record's, before
// the fills say which rows hold tokens) and dotted with the G queries from
// LDS. The online softmax then updates each head across the wavefront (base
// 2), and the value pass turns to lanes across channels, one token at a
// time. Rows are loaded whether or not they hold a token, so that no load
// waits for the fills; a row holding none enters the sums as zeros with
// weight 0. Page scores: eight lanes per page, each over D/8 channels, fp32
// products formed exactly in fp64 and added there, then summed over the
// eight lanes (a butterfly, so every lane of a page holds the same sum);
// each pass's loads go out one pass ahead, the first at entry.
// s_q: the unit's queries [GM][D] in LDS (heads past G zero), staged by the
// caller; s_p: this wavefront's [GM][64] weights in LDS; partial: the split's
// partial [G][D+2] (output, max, sum); score: the unit's [S] page scores, or
// [S][G] per-head bounds with the softmax aggregation.
template <int D, int GM>
__device__ __forceinline__ void f32_split(const LayerView& L, const StepIO& io, float scale_log2, int u, int split,
                                          const float* s_q, const float* s_kn, const float* s_vn, float (*s_p)[64],
                                          float* partial, double* score) {
    constexpr int DPL = D / 64;  // channels per lane in the value pass
    constexpr int CPP = D / 8;   // channels per lane in the page scores
    constexpr int VG = GM * DPL >= 32 ? 8 : 16;  // tokens whose value rows load together
    const int lane = threadIdx.x & 63;
    const int G = L.G, S = L.S, ps = L.ps;
    const size_t base = (size_t)u * S;
    const int t0 = split * L.bps * 32;
    const int t1 = max(t0, min(min(S * ps, 32 * L.nblk), t0 + L.bps * 32));
    const float* Ku = (const float*)L.K + (size_t)u * L.Lcap * D;
    const float* Vu = (const float*)L.V + (size_t)u * L.Lcap * D;
    const int32_t* fu = L.fill_att + base;  // fills the attention sees
    // the small reads first (loads complete in issue order): the unit record
    // and the first chunk's fills, then the key and value rows
    const int32_t* U4 = L.unit + (size_t)u * kUnitFields;
    const int ns = U4[kNextSlot], nf = U4[kNextFill];
    int f_pre = fu[min(t0 + lane, max(t1 - 1, 0)) / ps];

    // this lane's key row; the first chunk's now (rows below t1 lie inside
    // the unit's pool)
    float kr[D];
    auto load_key = [&](const float* kp) {
#pragma unroll
        for (int c = 0; c < D; c += 4) {
            const float4 x = *reinterpret_cast<const float4*>(kp + c);
            kr[c] = x.x;
            kr[c + 1] = x.y;
            kr[c + 2] = x.z;
            kr[c + 3] = x.w;
        }
    };
    load_key(Ku + (size_t)min(t0 + lane, max(t1 - 1, 0)) * D);
    // VPRE (head_dim 64, up to 8 head slots, where the registers allow): the
    // chunk's 64 value rows (one channel per lane) load together with its key
    // rows, before the fills and the unit record arrive, and the new token's
    // value is substituted afterwards
    constexpr bool VPRE = D == 64 && GM <= 8;
    float vpre[VPRE ? 64 : 1];
    auto load_vals = [&](int c0) {
        if constexpr (VPRE) {
#pragma unroll
            for (int e = 0; e < 64; ++e) vpre[e] = Vu[(size_t)min(c0 + e, max(t1 - 1, 0)) * D + lane];
        }
    };
    load_vals(t0);
    const float vn_lane = VPRE ? s_vn[lane] : 0.0f;
    // page state and representative keys of a score pass (pages pb .. pb+7,
    // clamped into the split's pages), loaded one pass ahead
    const int sl0 = min(S, (t0 + ps - 1) / ps), sl1 = min(S, (t1 + ps - 1) / ps);
    const int part = lane & 7, cb = part * CPP;
    float4 kx_nx[CPP / 4], kn_nx[CPP / 4];
    int st_nx = kFree;
    auto score_load = [&](int pb) {
        const size_t p = base + min(pb + (lane >> 3), sl1 - 1);
        st_nx = L.state[p];
#pragma unroll
        for (int c = 0; c < CPP; c += 4) {
            kx_nx[c / 4] = *reinterpret_cast<const float4*>((const float*)L.kmax + p * D + cb + c);
            kn_nx[c / 4] = *reinterpret_cast<const float4*>((const float*)L.kmin + p * D + cb + c);
        }
    };
    if (sl0 < sl1) score_load(sl0);
    const bool opened = nf == 0;
    const int row_new = ns * ps + nf;

    float m[GM], l[GM], acc[GM][DPL];
#pragma unroll
    for (int j = 0; j < GM; ++j) {
        m[j] = -INFINITY;
        l[j] = 0.0f;
#pragma unroll
        for (int i = 0; i < DPL; ++i) acc[j][i] = 0.0f;
    }
    for (int c0 = t0; c0 < t1; c0 += 64) {
        const int t = c0 + lane;
        if (c0 > t0) {  // later chunks' fills, key (and value) rows
            f_pre = fu[min(t, t1 - 1) / ps];
            load_key(Ku + (size_t)min(t, t1 - 1) * D);
            load_vals(c0);
        }
        bool valid = false;
        if (t < t1) {
            const int slot = t / ps;
            const int f = (slot == ns) ? nf + 1 : f_pre;
            valid = t - slot * ps < f;
        }
        const unsigned long long vmask = __ballot(valid);
        if (vmask == 0) continue;
        if (t == row_new) load_key(s_kn);
        // the heads' sums side by side (each in channel order)
        float sc[GM];
#pragma unroll
        for (int j = 0; j < GM; ++j) sc[j] = 0.0f;
#pragma unroll
        for (int c = 0; c < D; c += 4) {
#pragma unroll
            for (int j = 0; j < GM; ++j) {
                const float4 q4 = *reinterpret_cast<const float4*>(s_q + j * D + c);
                sc[j] = fmaf(q4.x, kr[c], sc[j]);
                sc[j] = fmaf(q4.y, kr[c + 1], sc[j]);
                sc[j] = fmaf(q4.z, kr[c + 2], sc[j]);
                sc[j] = fmaf(q4.w, kr[c + 3], sc[j]);
            }
        }
        // every head slot runs (those past G on zero queries, never written out)
#pragma unroll
        for (int j = 0; j < GM; ++j) {
            const float x = valid ? sc[j] * scale_log2 : -INFINITY;
            const float mx = wave_max_dpp(x);
            const float m_new = fmaxf(m[j], mx);  // finite: some lane holds a token
            const float alpha = __builtin_amdgcn_exp2f(m[j] - m_new);
            const float p = valid ? __builtin_amdgcn_exp2f(x - m_new) : 0.0f;
            l[j] = l[j] * alpha + wave_sum_dpp(p);
#pragma unroll
            for (int i = 0; i < DPL; ++i) acc[j][i] *= alpha;
            s_p[j][lane] = p;
            m[j] = m_new;
        }
        wave_lds_sync();
        if constexpr (VPRE) {
#pragma unroll
            for (int e = 0; e < 64; ++e) {
                const uint32_t keep = 0u - (uint32_t)((vmask >> e) & 1ull);  // all ones or zero
                const float v = __uint_as_float(__float_as_uint(c0 + e == row_new ? vn_lane : vpre[e]) & keep);
#pragma unroll
                for (int j = 0; j < GM; ++j) acc[j][0] = fmaf(s_p[j][e], v, acc[j][0]);
            }
        } else {
#pragma unroll
        for (int g0 = 0; g0 < 64; g0 += VG) {
            float vr[VG][DPL];
#pragma unroll
            for (int e = 0; e < VG; ++e) {
                const int tt = c0 + g0 + e;
                const uint32_t keep = 0u - (uint32_t)((vmask >> (g0 + e)) & 1ull);  // all ones or zero
                const float* vp = Vu + (size_t)min(tt, t1 - 1) * D;
#pragma unroll
                for (int i = 0; i < DPL; ++i) {
                    const float x = tt == row_new ? s_vn[lane + 64 * i] : vp[lane + 64 * i];
                    vr[e][i] = __uint_as_float(__float_as_uint(x) & keep);
                }
            }
#pragma unroll
            for (int e = 0; e < VG; ++e)
#pragma unroll
                for (int j = 0; j < GM; ++j) {
                    const float p = s_p[j][g0 + e];
#pragma unroll
                    for (int i = 0; i < DPL; ++i) acc[j][i] = fmaf(p, vr[e][i], acc[j][i]);
                }
        }
        }
        wave_lds_sync();  // the weights are read before the next chunk writes them
    }
#pragma unroll
    for (int j = 0; j < GM; ++j) {
        if (j >= G) break;
        float* pp = partial + (size_t)j * (D + 2);
#pragma unroll
        for (int i = 0; i < DPL; ++i) pp[lane + 64 * i] = acc[j][i];
        if (lane == 0) {
            pp[D] = m[j];
            pp[D + 1] = l[j];
        }
    }
    if (row_new >= t0 && row_new < t1) {  // append
        float* Kw = (float*)L.K + ((size_t)u * L.Lcap + row_new) * D;
        float* Vw = (float*)L.V + ((size_t)u * L.Lcap + row_new) * D;
        for (int c = lane; c < D; c += 64) {
            Kw[c] = s_kn[c];
            Vw[c] = s_vn[c];
        }
    }
    // page scores: pages whose first row lies in this split, eight at a time
    for (int pb = sl0; pb < sl1; pb += 8) {
        const int p = pb + (lane >> 3);
        const bool tail = p == ns;
        const bool act = p < sl1 && (tail || ranked(L, st_nx));
        float hi[CPP], lo[CPP];
#pragma unroll
        for (int c = 0; c < CPP; c += 4) {
            const float4 a = kx_nx[c / 4], b = kn_nx[c / 4];
            hi[c] = act ? a.x : 0.f, hi[c + 1] = act ? a.y : 0.f, hi[c + 2] = act ? a.z : 0.f;
            hi[c + 3] = act ? a.w : 0.f;
            lo[c] = act ? b.x : 0.f, lo[c + 1] = act ? b.y : 0.f, lo[c + 2] = act ? b.z : 0.f;
            lo[c + 3] = act ? b.w : 0.f;
        }
        if (pb + 8 < sl1) score_load(pb + 8);
        float* kx = (float*)L.kmax + (base + p) * D + cb;
        float* kn = (float*)L.kmin + (base + p) * D + cb;
        if (act && tail) {
#pragma unroll
            for (int c = 0; c < CPP; ++c) {
                const float x = s_kn[cb + c];
                hi[c] = opened ? x : fmaxf(hi[c], x);
                lo[c] = opened ? x : fminf(lo[c], x);
                kx[c] = hi[c];
                kn[c] = lo[c];
            }
        }
        double best = -INFINITY;
#pragma unroll 1
        for (int j = 0; j < G; ++j) {
            double a = 0.0;
#pragma unroll
            for (int c = 0; c < CPP; ++c) {
                const double qd = (double)s_q[j * D + cb + c];
                const double x = qd * (double)hi[c], y = qd * (double)lo[c];
                a += x > y ? x : y;
            }
            a += __shfl_xor(a, 1);
            a += __shfl_xor(a, 2);
            a += __shfl_xor(a, 4);
            best = a > best ? a : best;
            if (act && L.agg && part == 0) score[(size_t)p * G + j] = a;
        }
        if (act && !L.agg && part == 0) score[p] = best;
    }
}

// Step kernel, fp32 pools, split plan: one wavefront per (unit, split); the
// epilogue kernel merges the splits and runs the retention.
template <int D, int GM>
__global__ __launch_bounds__(64) void k_step_f32(LayerView L, StepIO io, float scale_log2) {
    __shared__ __align__(16) float s_q[GM * D];
    __shared__ __align__(16) float s_kn[D], s_vn[D];  // the new token's key and value
    __shared__ float s_p[GM][64];  // the chunk's weights, per head and token
    const int nsplit = L.nsplit;
    const int u = blockIdx.x / nsplit, split = blockIdx.x - (blockIdx.x / nsplit) * nsplit;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;
    const int G = L.G;
    const float* qg = (const float*)io.q + (size_t)u * G * D;
    for (int i = threadIdx.x; i < GM * D; i += 64) s_q[i] = i < G * D ? qg[i] : 0.0f;  // heads past G: zero
    for (int i = threadIdx.x; i < D; i += 64) {
        s_kn[i] = ((const float*)io.k_new)[(size_t)u * D + i];
        s_vn[i] = ((const float*)io.v_new)[(size_t)u * D + i];
    }
    __syncthreads();
    f32_split<D, GM>(L, io, scale_log2, u, split, s_q, s_kn, s_vn, s_p,
                     L.part + ((size_t)u * nsplit + split) * G * (D + 2), L.score + (size_t)u * L.S * (L.agg ? G : 1));
}

// head slots of the fp32 step kernel instance for a group of G heads
constexpr int f32_head_slots(int G) { return G <= 4 ? 4 : G <= 8 ? 8 : 16; }

// LDS of the fused fp32 step kernel with nw wavefronts: the queries, each
// wavefront's weights and partial, the slot arrays (score, state, ts, lid)
size_t f32_fused_lds(int GM, int G, int D, int S, int nw) {
    return (size_t)(GM + 2) * D * 4 + (size_t)nw * GM * 64 * 4 + (size_t)nw * G * (D + 2) * 4 + (size_t)S * 20;
}

// Step kernel, fp32 pools of head_dim 64, one workgroup per unit (L.nsplit
// <= 8 wavefronts, one per split): the splits' attention and page scores as
// above, into LDS;
// then, as the epilogue kernel does for split plans, the top-r refresh by the
// whole workgroup, the eviction by wavefront 0 while the others merge the
// wavefronts' partial outputs, and the state out. One launch per step.
template <int D, int GM>
__global__ __launch_bounds__(512) void k_step_f32_fused(LayerView L, StepIO io, float scale_log2, double r) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ RetShared ret;
    __shared__ int s_aux[260];
    const int u = blockIdx.x, tid = threadIdx.x, nth = blockDim.x, w = tid >> 6, nw = nth >> 6;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;
    const int G = L.G, S = L.S;
    float* s_q = reinterpret_cast<float*>(smem);                       // [GM][D]
    float* s_kn = s_q + GM * D;                                        // [D] the new token's key
    float* s_vn = s_kn + D;                                            // [D] and value
    float (*s_p)[64] = reinterpret_cast<float (*)[64]>(s_vn + D);      // [nw][GM][64]
    float* s_part = s_vn + D + (size_t)nw * GM * 64;                   // [nw][G][D+2]
    double* s_score = reinterpret_cast<double*>(s_part + (size_t)nw * G * (D + 2));  // [S] (8-byte aligned)
    int* s_state = reinterpret_cast<int*>(s_score + S);
    int* s_ts = s_state + S;
    int* s_lid = s_ts + S;
    const UnitRec ur = read_unit(L, u);
    load_slots(L, u, ur, s_score, s_state, s_ts, s_lid);  // every score +inf until its page is scored
    const float* qg = (const float*)io.q + (size_t)u * G * D;
    for (int i = tid; i < GM * D; i += nth) s_q[i] = i < G * D ? qg[i] : 0.0f;  // heads past G: zero
    for (int i = tid; i < D; i += nth) {
        s_kn[i] = ((const float*)io.k_new)[(size_t)u * D + i];
        s_vn[i] = ((const float*)io.v_new)[(size_t)u * D + i];
    }
    __syncthreads();
    f32_split<D, GM>(L, io, scale_log2, u, w, s_q, s_kn, s_vn, s_p + (size_t)w * GM, s_part + (size_t)w * G * (D + 2),
                     s_score);
    __syncthreads();
    refresh_block(L, ur, r, s_score, s_state, s_ts, s_aux, tid, nth, L.dbase);
    __syncthreads();
    if (tid < 64) evict_wave(L, ur, s_state, s_ts, s_lid, ret);
    for (int idx = tid; idx < G * D; idx += nth) {  // merge: out = sum_w 2^(M_w - M) O_w / sum_w 2^(M_w - M) L_w
        const int h = idx / D, c = idx - (idx / D) * D;
        float M = -INFINITY;
        for (int ww = 0; ww < nw; ++ww) M = fmaxf(M, s_part[((size_t)ww * G + h) * (D + 2) + D]);
        float O = 0.0f, Ls = 0.0f;
        for (int ww = 0; ww < nw; ++ww) {
            const float* pw = s_part + ((size_t)ww * G + h) * (D + 2);
            const float wt = (pw[D] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(pw[D] - M);
            O += wt * pw[c];
            Ls += wt * pw[D + 1];
        }
        ((float*)io.out)[((size_t)u * G + h) * D + c] = O / Ls;
    }
    __syncthreads();
    retention_store(L, io, u, ur, s_state, s_ts, s_lid, ret, tid, nth);
}

// Quest on the prompt pages (pools with a prompt region): for one unit, each
// kept prompt page's representative bound against the step's queries, max
// over the G heads of sum_c max(q_c kmax_c, q_c kmin_c) in fp64, channels
// summed in order; the topk pages of largest bound, ties to the lower slot,
// are attended. One thread per page reads the page's kmin/kmax rows with
// 16-byte loads and widens each key once for all heads; with q split into
// q+ = max(q, 0) and q- = min(q, 0), a channel's term is
// fma(q+, kmax, fma(q-, kmin, acc)): one of the two products is zero, which
// adds exactly, and the other is exact in fp64, so each bound rounds as the
// sequential sum does. Writes the fills the attention sees (0 for the other
// prompt pages) and the unit's block list: the prompt blocks holding a
// chosen page, ascending, then every block of the decode region. One
// workgroup per unit: 256 threads, 1024 when there are fewer units than CUs.
template <typename T>
__device__ __forceinline__ float vec_elem(const u32x4& x, int e);
template <>
__device__ __forceinline__ float vec_elem<uint16_t>(const u32x4& x, int e) { return bf2f(u16_at(x, e)); }
template <>
__device__ __forceinline__ float vec_elem<float>(const u32x4& x, int e) { return __uint_as_float(x[e]); }

// GQ: the query group size G, a compile-time constant so that the head loop
// unrolls into straight-line fused multiply-adds.

template <typename T, int GQ>
__global__ __launch_bounds__(1024) void k_prompt_select(LayerView L, StepIO io) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, nth = blockDim.x;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;
    constexpr int G = GQ;
    const int S = L.S, D = L.D, ps = L.ps, npr = L.dbase;
    const size_t base = (size_t)u * S;
    constexpr int V = 16 / sizeof(T);  // channels per 16-byte load
    double2* s_qpm = reinterpret_cast<double2*>(smem);                 // [G][D] (q+, q-)
    double* s_b = reinterpret_cast<double*>(s_qpm + (size_t)G * D);    // [npr] bounds
    int* s_sel = reinterpret_cast<int*>(s_b + npr);                    // [npr] chosen
    int* s_hist = s_sel + npr;  // [276] radix histogram, its pick, the count above theta, per-wavefront counts
    const int kp = L.unit[(size_t)u * kUnitFields + kPinnedPages];
    const T* qg = (const T*)io.q + (size_t)u * G * D;
    for (int i = tid; i < G * D; i += nth) {
        const double q = (double)to_f(qg[i]);
        s_qpm[i] = make_double2(q > 0.0 ? q : 0.0, q < 0.0 ? q : 0.0);
    }
    __syncthreads();
    const bool all = kp <= L.topk;
    for (int p = tid; p < kp && !all; p += nth) {
        const T* kx = (const T*)L.kmax + (base + p) * D;
        const T* kn = (const T*)L.kmin + (base + p) * D;
        double acc[G];
#pragma unroll
        for (int j = 0; j < G; ++j) acc[j] = 0.0;
#pragma unroll 4
        for (int c = 0; c < D; c += V) {
            const u32x4 xv = ld4(kx + c), nv = ld4(kn + c);
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const double hi = (double)vec_elem<T>(xv, e), lo = (double)vec_elem<T>(nv, e);
#pragma unroll
                for (int j = 0; j < G; ++j) {
                    const double2 qpm = s_qpm[j * D + c + e];
                    acc[j] = fma(qpm.x, hi, fma(qpm.y, lo, acc[j]));
                }
            }
        }
        double best = -INFINITY;
#pragma unroll
        for (int j = 0; j < G; ++j) best = fmax(best, acc[j]);
        s_b[p] = best;
    }
    __syncthreads();
    // the topk pages of largest bound, ties to the lower slot. Up to 256
    // pages, each page is ranked against all others; beyond (the count is
    // quadratic in the pages), theta, the topk-th largest bound (counted with
    // multiplicity), by a radix select, then every page above it and, of
    // those equal to it, the lowest slots, as many as are left (a prefix
    // count in slot order): the same pages.
    if (all || kp <= 256) {
        for (int p = tid; p < npr; p += nth) {
            bool sel = p < kp;
            if (sel && !all) {
                const double bp = s_b[p];
                int above = 0;
                for (int o = 0; o < kp; ++o) above += (s_b[o] > bp || (s_b[o] == bp && o < p)) ? 1 : 0;
                sel = above < L.topk;
            }
            s_sel[p] = sel ? 1 : 0;
        }
    } else {
        const double theta = kth_largest_f64_wg(s_b, kp, L.topk, s_hist, tid, nth);
        if (tid == 0) s_hist[258] = 0;
        __syncthreads();
        int gt = 0;
        for (int p = tid; p < kp; p += nth) gt += s_b[p] > theta ? 1 : 0;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) gt += __shfl_xor(gt, off);
        if (lane == 0 && gt) atomicAdd(&s_hist[258], gt);
        __syncthreads();
        const int need = L.topk - s_hist[258], w = tid >> 6, nw = nth >> 6;
        int run = 0;  // tied pages in the slots before this chunk
        for (int c0 = 0; c0 < kp; c0 += nth) {
            const int p = c0 + tid;
            const bool eq = p < kp && s_b[p] == theta;
            const unsigned long long m = __ballot(eq);
            if (lane == 0) s_hist[259 + w] = __popcll(m);
            __syncthreads();
            int before = run + __popcll(m & ((1ull << lane) - 1ull)), tot = 0;
            for (int ww = 0; ww < nw; ++ww) {
                const int cw = s_hist[259 + ww];
                tot += cw;
                before += ww < w ? cw : 0;
            }
            if (p < kp) s_sel[p] = (s_b[p] > theta || (eq && before < need)) ? 1 : 0;
            run += tot;
            __syncthreads();
        }
        for (int p = kp + tid; p < npr; p += nth) s_sel[p] = 0;
    }
    __syncthreads();
    for (int p = tid; p < npr; p += nth) L.fill_att[base + p] = s_sel[p] ? L.fill[base + p] : 0;
    for (int s = npr + tid; s < S; s += nth) L.fill_att[base + s] = L.fill[base + s];
    __syncthreads();
    if (tid < 64) {
        const int nbp = npr * ps / 32;  // prompt blocks (the region is a whole number of blocks)
        int32_t* bl = L.blist + (size_t)u * L.lcap_blk;
        int cnt = 0;
        for (int c0 = 0; c0 < nbp; c0 += 64) {
            const int b = c0 + lane;
            bool any = false;
            if (b < nbp)
                for (int s = 32 * b / ps; s <= (32 * b + 31) / ps; ++s) any = any || s_sel[s] != 0;
            const unsigned long long m = __ballot(any);
            if (any) bl[cnt + __popcll(m & ((1ull << lane) - 1ull))] = b;
            cnt += __popcll(m);
        }
        for (int b = nbp + lane; b < L.nblk; b += 64) bl[cnt + b - nbp] = b;
        if (lane == 0) {
            L.bcnt[2 * u] = cnt;
            L.bcnt[2 * u + 1] = cnt + max(0, L.nblk - nbp);
        }
    }
}

// The kept prompt pages' bound intervals (prompt_bounds) into L.pivl, for
// units too few to fill the chip: one wavefront per L.pchunk pages of a
// unit, so that the pages' representative keys stream through many CUs;
// nothing for units with no more kept pages than topk.
template <int D>
__global__ __launch_bounds__(64) void k_prompt_intervals(LayerView L, StepIO io) {
    constexpr int KS = D / 32;
    const int nch = (L.dbase + L.pchunk - 1) / L.pchunk;
    const int u = blockIdx.x / nch, ch = blockIdx.x - u * nch;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;
    const int kp = L.unit[(size_t)u * kUnitFields + kPinnedPages], p0 = ch * L.pchunk;
    if (kp <= L.topk || p0 >= kp) return;
    const int n = min(L.pchunk, kp - p0), lane = threadIdx.x, grp = lane >> 4, col = lane & 15;
    const uint16_t* qg = (const uint16_t*)io.q + (size_t)u * L.G * D;
    bf16x8 qv[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const u32x4 x = (col < L.G) ? ld4(qg + (size_t)col * D + 32 * ks + 8 * grp) : u32x4{0u, 0u, 0u, 0u};
        qv[ks] = __builtin_bit_cast(bf16x8, x);
    }
    float* lo = L.pivl + (size_t)u * L.dbase + p0;
    prompt_bounds<D, 1, false>(L, (size_t)u * L.S + p0, n, qv, lo, lo + (size_t)L.U * L.dbase, [] {});
}

// The same selection for bf16 pools, on the MFMA: each kept prompt page's
// bound as an interval (prompt_bounds), lo_cut the topk-th largest lower end,
// and the candidates, the pages whose upper end reaches lo_cut; at least
// topk pages have bounds >= lo_cut, so every other page ranks below all of
// them. Only the candidates' bounds are taken exactly (fp64, as the decode
// pages' scores), and the topk among them, ties to the lower slot, are the
// chosen pages. Then the fills and the block list, as above, the list's
// positions by a prefix count over the whole workgroup. One workgroup of
// NW wavefronts per unit. With L.pchunk > 0 the intervals come from
// k_prompt_intervals, launched just before.
template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void k_prompt_select_mfma(LayerView L, StepIO io) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ int s_lo, s_ncand, s_wc[NW];
    constexpr int KS = D / 32, NT = NW * 64;
    const int u = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6, grp = lane >> 4, col = lane & 15;
    if (io.active != nullptr && io.active[u / L.nkv] == 0) return;
    const int G = L.G, S = L.S, ps = L.ps, npr = L.dbase;
    const size_t base = (size_t)u * S;
    float* s_qf = reinterpret_cast<float*>(smem);     // [G][qpad_row(D)] q in fp32 (a multiple of 16 bytes)
    float* s_plo = s_qf + (size_t)G * qpad_row(D);    // [npr] bound intervals (16-byte reads of s_plo)
    float* s_phi = s_plo + npr;
    double* s_ex = reinterpret_cast<double*>(s_phi + npr);  // [npr] candidates' exact bounds
    int* s_cand = reinterpret_cast<int*>(s_ex + npr);       // [npr] candidates
    int* s_sel = s_cand + npr;                          // [npr] chosen
    int* s_hist = s_sel + npr;                          // [258] radix histogram and its pick
    const int kp = L.unit[(size_t)u * kUnitFields + kPinnedPages];
    const bool all = kp <= L.topk;
    // lane (grp, col < G): head col's channels 32 ks + 8 grp .. +7, the MFMA's query operands
    const uint16_t* qg = (const uint16_t*)io.q + (size_t)u * G * D;
    bf16x8 qv[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const u32x4 x = (col < G) ? ld4(qg + (size_t)col * D + 32 * ks + 8 * grp) : u32x4{0u, 0u, 0u, 0u};
        qv[ks] = __builtin_bit_cast(bf16x8, x);
    }
    for (int p = tid; p < npr; p += NT) s_sel[p] = p < kp ? 1 : 0;
    if (tid == 0) {
        s_lo = 0x7FFFFFFF;
        s_ncand = 0;
    }
    if (!all) {
        // q in fp32 for the exact bounds, the wavefronts taking turns over ks
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            if (ks % NW == w && col < G) {
                const u32x4 x = __builtin_bit_cast(u32x4, qv[ks]);
                float* d = s_qf + qpad_index<D>(col * D + 32 * ks + 8 * grp);
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    d[2 * h] = __uint_as_float(x[h] << 16);
                    d[2 * h + 1] = __uint_as_float(x[h] & 0xFFFF0000u);
                }
            }
        }
        if (L.pchunk > 0) {
            const float* glo = L.pivl + (size_t)u * npr;
            const float* ghi = glo + (size_t)L.U * npr;
            for (int p = tid; p < kp; p += NT) {
                s_plo[p] = glo[p];
                s_phi[p] = ghi[p];
            }
        } else {
            prompt_bounds<D, NW, false>(L, base, kp, qv, s_plo, s_phi, [] {});
        }
    }
    __syncthreads();
    if (!all) {
        float lo_cut;
        if (kp > 256) {  // (the count is quadratic in the pages)
            lo_cut = kth_largest_wg<NT>(s_plo, kp, L.topk, s_hist, tid);
        } else {
            const int kp4 = kp & ~3;
            for (int p = tid; p < kp; p += NT) {
                const float lp = s_plo[p];
                int above = 0;  // lower ends above p's: four per 16-byte read, then the last few
#pragma unroll 4
                for (int o = 0; o < kp4; o += 4) {
                    const float4 x = *reinterpret_cast<const float4*>(s_plo + o);
                    above += (x.x > lp ? 1 : 0) + (x.y > lp ? 1 : 0) + (x.z > lp ? 1 : 0) + (x.w > lp ? 1 : 0);
                }
                for (int o = kp4; o < kp; ++o) above += s_plo[o] > lp ? 1 : 0;
                if (above < L.topk) atomicMin(&s_lo, float_order(lp));
            }
            __syncthreads();
            lo_cut = order_float(s_lo);
        }
        for (int p = tid; p < kp; p += NT) {
            if (s_phi[p] >= lo_cut) s_cand[atomicAdd(&s_ncand, 1)] = p;
            else s_sel[p] = 0;
        }
        __syncthreads();
        // exactly topk candidates: they are the top k; more: their bounds in
        // fp64, eight lanes per page, and the topk of those
        const int nc = s_ncand;
        if (nc > L.topk) {
            for (int c0 = 8 * w; c0 < nc; c0 += 8 * NW) {
                const int c = c0 + (lane >> 3);
                const bool act = c < nc;
                const int p = act ? s_cand[c] : 0;
                ScoreFrag<D> f;
                score_issue<D>(L, u, p, lane & 7, act, f);
                const double sc = score_finish<D>(L, u, p, lane & 7, act, f, false, false, nullptr, s_qf, nullptr);
                if (act && (lane & 7) == 0) s_ex[c] = sc;
            }
            __syncthreads();
            for (int c = tid; c < nc; c += NT) {
                const int p = s_cand[c];
                const double e = s_ex[c];
                int above = 0;
                for (int o = 0; o < nc; ++o) {
                    const double x = s_ex[o];
                    above += (x > e || (x == e && s_cand[o] < p)) ? 1 : 0;
                }
                if (above >= L.topk) s_sel[p] = 0;
            }
        }
    }
    __syncthreads();
    for (int p = tid; p < npr; p += NT) L.fill_att[base + p] = s_sel[p] ? L.fill[base + p] : 0;
    for (int sl = npr + tid; sl < S; sl += NT) L.fill_att[base + sl] = L.fill[base + sl];
    // the prompt blocks holding a chosen page, ascending (a block's place: the
    // chosen blocks before it, in its wavefront and in the ones before), then
    // every block of the decode region
    const int nbp = npr * ps / 32;
    int32_t* bl = L.blist + (size_t)u * L.lcap_blk;
    int run = 0;
    for (int c0 = 0; c0 < nbp; c0 += NT) {
        const int bb = c0 + tid;
        bool any = false;
        if (bb < nbp)
            for (int sl = 32 * bb / ps; sl <= (32 * bb + 31) / ps; ++sl) any = any || s_sel[sl] != 0;
        const unsigned long long m = __ballot(any);
        if (lane == 0) s_wc[w] = __popcll(m);
        __syncthreads();
        int before = run + __popcll(m & ((1ull << lane) - 1ull)), tot = 0;
#pragma unroll
        for (int ww = 0; ww < NW; ++ww) {
            tot += s_wc[ww];
            before += ww < w ? s_wc[ww] : 0;
        }
        if (any) bl[before] = bb;
        run += tot;
        __syncthreads();
    }
    for (int b = nbp + tid; b < L.nblk; b += NT) bl[run + b - nbp] = b;
    if (tid == 0) {
        L.bcnt[2 * u] = run;
        L.bcnt[2 * u + 1] = run + max(0, L.nblk - nbp);
    }
}

// Epilogue kernel of the split path: the retention policy on the scores the
// step kernel wrote, and the merge of the splits' partial attention
// (out = sum_s 2^(M_s - M) O_s / sum_s 2^(M_s - M) L_s); then the state goes
// out. One workgroup per decision: L.hgrp units (the KV heads of a sequence
// when they share one page table, whose slot states are then identical), a
// page's score aggregating the bounds of all their heads. The refresh runs
// on the whole workgroup; wavefront 0 then evicts while the others start
// the merge. merge 0: the step kernel wrote the outputs (bf16, one
// workgroup per unit).
template <typename T>
__global__ __launch_bounds__(1024) void k_epilogue(LayerView L, StepIO io, double r, int merge) {
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ RetShared ret;
    __shared__ int s_aux[260];
    const int S = L.S, G = L.G, D = L.D, nsplit = L.nsplit, nu = L.hgrp;
    const int tid = threadIdx.x, nth = blockDim.x;
    double* s_score = reinterpret_cast<double*>(smem);
    double* s_mz = s_score + S;  // [nu*G][2], softmax aggregation only
    float* s_ml = reinterpret_cast<float*>(s_mz + (L.agg ? 2 * (size_t)nu * G : 0));  // [nsplit][G][2], merge
    float* s_den = s_ml + (merge ? 2 * (size_t)nsplit * G : 0);                       // [G], merge
    int* s_state = reinterpret_cast<int*>(s_den + (merge ? G : 0));
    int* s_ts = s_state + S;
    int* s_lid = s_ts + S;
    const int u0 = blockIdx.x * nu;
    if (io.active != nullptr && io.active[u0 / L.nkv] == 0) return;
    const size_t base = (size_t)u0 * S;
    // The first pass's reads go out together with the slots': the page
    // score of slot tid (max over the units; read whether or not the page
    // turns out to be ranked) and the first unit's running maximum and sum
    // of item tid of the merge.
    double sc_first = -INFINITY;
    if (!L.agg && tid < S) {
        sc_first = L.score[base + tid];
#pragma unroll 8
        for (int h = 1; h < nu; ++h) sc_first = fmax(sc_first, L.score[base + (size_t)h * S + tid]);
    }
    float m_first = 0.0f, l_first = 0.0f;
    if (merge && tid < nsplit * G) {
        const float* pf = L.part + (size_t)u0 * nsplit * G * (D + 2) + (size_t)tid * (D + 2);
        m_first = pf[D];
        l_first = pf[D + 1];
    }
    const UnitRec ur = read_unit(L, u0);
    load_slots(L, u0, ur, s_score, s_state, s_ts, s_lid);
    __syncthreads();
    if (!L.agg) {
        if (tid < S && ranked(L, s_state[tid])) s_score[tid] = sc_first;
        for (int s = tid + nth; s < S; s += nth)
            if (ranked(L, s_state[s])) {
                double best = L.score[base + s];
#pragma unroll 8
                for (int h = 1; h < nu; ++h) best = fmax(best, L.score[base + (size_t)h * S + s]);
                s_score[s] = best;
            }
    }
    __syncthreads();
    if (L.agg) softmax_sum_block(L, L.score + base * G, nu, s_state, s_score, s_mz, tid, nth);
    refresh_block(L, ur, r, s_score, s_state, s_ts, s_aux, tid, nth, L.dbase);
    __syncthreads();
    if (tid < 64) evict_wave(L, ur, s_state, s_ts, s_lid, ret);
    for (int uh = 0; merge && uh < nu; ++uh) {
        const int u = u0 + uh;
        const float* pu = L.part + (size_t)u * nsplit * G * (D + 2);
        // every split's running max and sum, then per head the weights' sum
        if (uh == 0 && tid < nsplit * G) {
            s_ml[2 * tid] = m_first;
            s_ml[2 * tid + 1] = l_first;
        }
        for (int i = uh == 0 ? tid + nth : tid; i < nsplit * G; i += nth) {
            s_ml[2 * i] = pu[(size_t)i * (D + 2) + D];
            s_ml[2 * i + 1] = pu[(size_t)i * (D + 2) + D + 1];
        }
        __syncthreads();
        for (int h = tid; h < G; h += nth) {
            float M = -INFINITY;
            for (int s = 0; s < nsplit; ++s) M = fmaxf(M, s_ml[2 * (s * G + h)]);
            float Ls = 0.0f;
            for (int s = 0; s < nsplit; ++s) {
                const float ms = s_ml[2 * (s * G + h)];
                const float wt = (ms == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(ms - M);
                s_ml[2 * (s * G + h)] = wt;  // the split's weight replaces its max
                Ls += wt * s_ml[2 * (s * G + h) + 1];
            }
            s_den[h] = Ls;
        }
        __syncthreads();
        for (int idx = tid; idx < G * D; idx += nth) {
            const int h = idx / D, c = idx - (idx / D) * D;
            float O = 0.0f;
#pragma unroll 4
            for (int s = 0; s < nsplit; ++s) O += s_ml[2 * (s * G + h)] * pu[((size_t)s * G + h) * (D + 2) + c];
            ((T*)io.out)[((size_t)u * G + h) * D + c] = from_f<T>(O / s_den[h]);
        }
        __syncthreads();
    }
    __syncthreads();
    for (int uh = 0; uh < nu; ++uh)
        retention_store(L, io, u0 + uh, ur, s_state, s_ts, s_lid, ret, tid, nth);
}

inline unsigned grid1d(size_t n, int block) { return (unsigned)((n + block - 1) / block); }

// LDS of the step kernel: the queries in fp32, the attention wavefronts'
// partial outputs, the fused epilogue's slot arrays (with the per-head
// bounds of the softmax aggregation), and a block list
size_t step_lds(int G, int D, int S, int NW, bool fused, int agg, int list_ints) {
    size_t b = (size_t)4 * G * qpad_row(D) + (size_t)NW * G * (D + 4) * 4;
    if (fused) b += (size_t)S * 20 + (agg ? (size_t)S * G * 8 + (size_t)G * 16 : 0);
    return b + (size_t)list_ints * 4;
}

template <int D, int NW, bool AGG, int LM, bool NT = false>
void launch_step_inst(const LayerView& L, const StepIO& io, const StepPlan& pl, float sl2, double r,
                      hipStream_t s) {
    hipLaunchKernelGGL((k_step_bf16<D, NW, AGG, LM, NT>), dim3((unsigned)(L.U * pl.nsplit)), dim3(NW * 64),
                       pl.lds, s, L, io, sl2, r, pl.fused ? 1 : 0);
}

template <int D, int NW>
hipError_t launch_step_bf16(const LayerView& L, const StepIO& io, const StepPlan& pl, float sl2, double r,
                            hipStream_t s) {
    const bool list = L.topk >= 0;
    if (L.agg) {
        if (list && L.nt) launch_step_inst<D, NW, true, 1, true>(L, io, pl, sl2, r, s);
        else if (list) launch_step_inst<D, NW, true, 1>(L, io, pl, sl2, r, s);
        else if (L.nt) launch_step_inst<D, NW, true, 0, true>(L, io, pl, sl2, r, s);
        else launch_step_inst<D, NW, true, 0>(L, io, pl, sl2, r, s);
    } else {
        if (pl.select_in_step && L.nt) launch_step_inst<D, NW, false, 2, true>(L, io, pl, sl2, r, s);
        else if (pl.select_in_step) launch_step_inst<D, NW, false, 2>(L, io, pl, sl2, r, s);
        else if (list && L.nt) launch_step_inst<D, NW, false, 1, true>(L, io, pl, sl2, r, s);
        else if (list) launch_step_inst<D, NW, false, 1>(L, io, pl, sl2, r, s);
        else if (L.nt) launch_step_inst<D, NW, false, 0, true>(L, io, pl, sl2, r, s);
        else launch_step_inst<D, NW, false, 0>(L, io, pl, sl2, r, s);
    }
    return hipGetLastError();
}

template <int D, int NW>
hipError_t allow_lds_all(int bytes) {
    hipError_t e = hipSuccess;
    auto set = [&](const void* f) {
        hipError_t r = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (r != hipSuccess) e = r;
    };
    set((const void*)k_step_bf16<D, NW, false, 0>);
    set((const void*)k_step_bf16<D, NW, true, 0>);
    set((const void*)k_step_bf16<D, NW, false, 1>);
    set((const void*)k_step_bf16<D, NW, true, 1>);
    set((const void*)k_step_bf16<D, NW, false, 2>);
    set((const void*)k_step_bf16<D, NW, false, 0, true>);
    set((const void*)k_step_bf16<D, NW, false, 2, true>);
    set((const void*)k_step_bf16<D, NW, true, 0, true>);
    set((const void*)k_step_bf16<D, NW, false, 1, true>);
    set((const void*)k_step_bf16<D, NW, true, 1, true>);
    return e;
}

}  // namespace

// ---------------------------------------------------------------------------

// Blocks per wavefront up to which one fused workgroup per unit is chosen
// over a split (measured at batch 1 and 4, 32 blocks per unit over 8
// wavefronts: 14.6 against 19.2 us and 15.9 against 19.7 us per step), and
// up to kFusedBlocksPerWaveFewSlots with at most kFewSlots slots, where the
// fused workgroup's retention (one wavefront counting over all slots) is
// short: 64 blocks and 64 slots at batch 1, 4 and 8, the fused kernel
// 17.1, 17.4 and 18.0 us against 17.6, 18.6 and 20.4 us for the split
// path's two kernels before their second launch; with 128 slots (page 16)
// fused took 22.0 against 20.3 us per step at batch 4.
constexpr int kFusedBlocksPerWave = 6;
constexpr int kFusedBlocksPerWaveFewSlots = 8;
constexpr int kFewSlots = 64;
// With a prompt region and fewer units than CUs, fused up to this many
// attended blocks per wavefront and prompt pages (batch 1 and 8, 128 prompt
// pages, 72 attended blocks over 8 wavefronts: 30.3 against 36.2 and 32.2
// against 36.2 us per step; batch 4, 512 pages, 80 blocks: 44.0 against
// 54.4 us, the fused kernel 40.1 us and the split path's four kernels 37.5
// to 39.1 us before their launch gaps; at 1024 prompt pages the fused
// workgroup's own bound intervals cost more than the split path's
// kernels: 68.8 against 45.9 us at batch 1).
constexpr int kFusedPromptBlocksPerWave = 12;
constexpr int kFusedPromptPages = 512;

// Workgroups of 2 wavefronts, four per CU, from this many units on when a
// unit's step attends at most kSmallWorkBlocks blocks (same box, batch 128,
// page 32: L 512 45.1 -> 42.7 us, L 512 plus the top 8 prompt pages 114.4 ->
// 101.8 us; L 2048, 64 blocks, 170.1 -> 173.4 us, so longer pools keep 4).
constexpr int kSmallWorkUnits = 1024;
constexpr int kSmallWorkBlocks = 32;

StepPlan plan_step(int U, int G, int D, int S, int Lcap, int ps, int work_blocks, bool bf16, int agg,
                   bool grouped, int list_ints, int split_override, int npr) {
    (void)ps;
    StepPlan pl{};
    const int nblk = Lcap / kBlockTokens;
    int want;
    if (!bf16) {
        pl.waves = 1;
        want = split_override > 0 ? split_override : (nblk + 1) / 2;
    } else {
        pl.waves = 2;
        for (int nw : {8, 4, 2}) {
            if (step_lds(G, D, S, nw, false, agg, list_ints) <= kMaxLds) {
                pl.waves = nw;
                break;
            }
        }
        // two or more units per CU: workgroups of 4 wavefronts, two per CU,
        // so that one unit's serial phases (staging, selection, retention)
        // overlap another's streaming
        if (split_override <= 0 && !grouped && U >= 512 && pl.waves == 8 &&
            2 * step_lds(G, D, S, 4, true, agg, list_ints) <= kMaxLds)
            pl.waves = 4;
        // four or more units per CU, each with little to stream: four
        // workgroups per CU overlap more units' serial phases
        if (split_override <= 0 && !grouped && U >= kSmallWorkUnits && work_blocks <= kSmallWorkBlocks &&
            pl.waves == 4 && 4 * step_lds(G, D, S, 2, true, agg, list_ints) <= kMaxLds)
            pl.waves = 2;
        if (split_override > 0) {
            want = split_override;
        } else if (!grouped &&
                   (nblk <= kFusedBlocksPerWave * pl.waves ||
                    (S <= kFewSlots && nblk <= kFusedBlocksPerWaveFewSlots * pl.waves)) &&
                   step_lds(G, D, S, pl.waves, true, agg, list_ints) <= kMaxLds) {
            // few blocks per wavefront: one workgroup per unit, which also runs
            // the epilogue, beats spreading the unit over more CUs and paying a
            // second launch (about 10 us) for the merge
            want = 1;
        } else if (!grouped && list_ints > 0 && !agg && U < 256 && npr <= kFusedPromptPages &&
                   work_blocks <= kFusedPromptBlocksPerWave * pl.waves &&
                   step_lds(G, D, S, pl.waves, true, agg, list_ints) <= kMaxLds) {
            // a short prompt region: the fused workgroup chooses its prompt
            // pages itself and attends the chosen blocks and the decode ones,
            // which saves the selection kernel's launch as well
            want = 1;
        } else {
            // one workgroup per CU over the 256 CUs
            const double per_wave = fmax(1.0, (double)U * nblk / (256.0 * pl.waves));
            want = (int)ceil(nblk / (pl.waves * per_wave) - 1e-9);
        }
    }
    want = want < 1 ? 1 : want;
    want = want > kMaxSplits ? kMaxSplits : want;
    want = want > nblk ? nblk : want;
    pl.bps = (nblk + want - 1) / want;
    pl.nsplit = (nblk + pl.bps - 1) / pl.bps;
    if (bf16) {
        pl.fused = !grouped && pl.nsplit == 1 && step_lds(G, D, S, pl.waves, true, agg, list_ints) <= kMaxLds;
        pl.lds = step_lds(G, D, S, pl.waves, pl.fused, agg, list_ints);
    } else {
        // fp32: one workgroup per unit with a wavefront per split (up to 8,
        // two per SIMD at the kernel's registers), which then runs the
        // epilogue itself; the softmax aggregation, the sequence scope, a
        // prompt region and head_dim 128 (whose key rows would spill the
        // fused kernel's registers) keep the epilogue kernel
        pl.fused = D == 64 && !grouped && !agg && list_ints == 0 && pl.nsplit <= 8 &&
                   f32_fused_lds(f32_head_slots(G), G, D, S, pl.nsplit) <= kMaxLds;
        pl.lds = pl.fused ? f32_fused_lds(f32_head_slots(G), G, D, S, pl.nsplit) : 0;
    }
    // a fused workgroup covers its unit, so it can choose the prompt pages
    // itself (the softmax aggregation keeps the selection kernel)
    pl.select_in_step = bf16 && pl.fused && list_ints > 0 && !agg;
    return pl;
}

hipError_t allow_large_lds() {
    const int bytes = (int)kMaxLds;
    hipError_t e = hipSuccess;
    for (hipError_t r : {allow_lds_all<128, 8>(bytes), allow_lds_all<128, 4>(bytes), allow_lds_all<128, 2>(bytes),
                         allow_lds_all<64, 8>(bytes), allow_lds_all<64, 4>(bytes), allow_lds_all<64, 2>(bytes)})
        if (r != hipSuccess) e = r;
    for (const void* f : {(const void*)k_step_f32_fused<64, 4>, (const void*)k_step_f32_fused<64, 8>,
                          (const void*)k_step_f32_fused<64, 16>}) {
        hipError_t r = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
        if (r != hipSuccess) e = r;
    }

    return e;
}

template <typename T, int GQ>
void launch_select_g(const LayerView& L, const StepIO& io, size_t shm, hipStream_t stream) {
    // fewer units than CUs: a unit's pages over more threads
    hipLaunchKernelGGL((k_prompt_select<T, GQ>), dim3(L.U), dim3(L.U < 256 ? 1024 : 256), shm, stream, L, io);
}

template <typename T, int... GS>
void launch_select_t(const LayerView& L, const StepIO& io, size_t shm, hipStream_t stream,
                     std::integer_sequence<int, GS...>) {
    ((L.G == GS + 1 ? launch_select_g<T, GS + 1>(L, io, shm, stream) : void()), ...);
}

template <int D>
void launch_select_mfma(const LayerView& L, const StepIO& io, hipStream_t stream) {
    // q in fp32 (padded rows), per prompt slot the interval, the exact bound,
    // the candidate and the chosen flag, and the radix histogram
    const size_t shm = (size_t)L.G * qpad_row(D) * 4 + (size_t)L.dbase * 24 + 258 * 4;
    if (L.pchunk > 0) {
        const int nch = (L.dbase + L.pchunk - 1) / L.pchunk;
        hipLaunchKernelGGL((k_prompt_intervals<D>), dim3(L.U * nch), dim3(64), 0, stream, L, io);
    }
    // fewer units than CUs: 8 wavefronts per unit; four units per CU and
    // more: 2, so that more units are resident at once
    if (L.U < 256)
        hipLaunchKernelGGL((k_prompt_select_mfma<D, 8>), dim3(L.U), dim3(512), shm, stream, L, io);
    else if (L.U < 1024)
        hipLaunchKernelGGL((k_prompt_select_mfma<D, 4>), dim3(L.U), dim3(256), shm, stream, L, io);
    else
        hipLaunchKernelGGL((k_prompt_select_mfma<D, 2>), dim3(L.U), dim3(128), shm, stream, L, io);
}

hipError_t launch_prompt_select(const LayerView& L, const StepIO& io, hipStream_t stream) {
    if (L.bf16) {
        if (L.D == 128)
            launch_select_mfma<128>(L, io, stream);
        else
            launch_select_mfma<64>(L, io, stream);
        return hipGetLastError();
    }
    // q split in two (16 B per element), the bounds and the chosen flags, the
    // radix histogram and its counts
    const size_t shm = (size_t)L.G * L.D * 16 + (size_t)L.dbase * 12 + 276 * 4;
    launch_select_t<float>(L, io, shm, stream, std::make_integer_sequence<int, 16>{});
    return hipGetLastError();
}

hipError_t launch_prefill(const LayerView& L, const void* k, const void* v, const PrefillIn& in, int max_tok,
                          hipStream_t stream) {
    hipLaunchKernelGGL(k_prefill_meta, dim3(L.U), dim3(256), 0, stream, L, in);
    if (max_tok > 0) {
        if (L.bf16) {
            const size_t n = (size_t)L.U * max_tok * (L.D / 8) + (size_t)L.U * ((max_tok + 7) / 8) * L.D;
            if (L.D == 128)
                hipLaunchKernelGGL(k_prefill_bf16<128>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const uint16_t*)k, (const uint16_t*)v, in, max_tok);
            else
                hipLaunchKernelGGL(k_prefill_bf16<64>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const uint16_t*)k, (const uint16_t*)v, in, max_tok);
        } else {
            const size_t n = (size_t)L.U * max_tok * (L.D / 4);
            hipLaunchKernelGGL(k_prefill_f32, dim3(grid1d(n, 256)), dim3(256), 0, stream, L, (const float*)k,
                               (const float*)v, in, max_tok);
        }
        if (L.rank_pinned || L.topk >= 0) {
            const int max_pages = (max_tok + L.ps - 1) / L.ps;
            const size_t n = (size_t)L.U * max_pages * L.D;
            if (L.bf16)
                hipLaunchKernelGGL(k_prefill_rep<uint16_t>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const uint16_t*)k, in, max_pages);
            else
                hipLaunchKernelGGL(k_prefill_rep<float>, dim3(grid1d(n, 256)), dim3(256), 0, stream, L,
                                   (const float*)k, in, max_pages);
        }
    }
    return hipGetLastError();
}

// fp32 step kernel with room for GM >= G query heads (the head loops unroll
// GM times: a small bound keeps the kernel's code small)
template <int D, int GM>
void launch_step_f32_gm(const LayerView& L, const StepIO& io, const StepPlan& pl, float sl2, double r, hipStream_t s) {
    if constexpr (D == 64) {
        if (pl.fused) {
            hipLaunchKernelGGL((k_step_f32_fused<D, GM>), dim3((unsigned)L.U), dim3(64 * pl.nsplit), pl.lds, s, L, io,
                               sl2, r);
            return;
        }
    }
    hipLaunchKernelGGL((k_step_f32<D, GM>), dim3((unsigned)(L.U * pl.nsplit)), dim3(64), 0, s, L, io, sl2);
}

template <int D>
void launch_step_f32(const LayerView& L, const StepIO& io, const StepPlan& pl, float sl2, double r, hipStream_t s) {
    if (L.G <= 4) launch_step_f32_gm<D, 4>(L, io, pl, sl2, r, s);
    else if (L.G <= 8) launch_step_f32_gm<D, 8>(L, io, pl, sl2, r, s);
    else launch_step_f32_gm<D, 16>(L, io, pl, sl2, r, s);
}

hipError_t launch_step(const LayerView& L, const StepIO& io, const StepPlan& pl, double r, hipStream_t s) {
    const float sl2 = (float)(1.4426950408889634 / sqrt((double)L.D));
    if (!L.bf16) {
        if (L.D == 128) launch_step_f32<128>(L, io, pl, sl2, r, s);
        else launch_step_f32<64>(L, io, pl, sl2, r, s);
        return hipGetLastError();
    }
    if (L.D == 128) {
        switch (pl.waves) {
            case 8: return launch_step_bf16<128, 8>(L, io, pl, sl2, r, s);
            case 4: return launch_step_bf16<128, 4>(L, io, pl, sl2, r, s);
            default: return launch_step_bf16<128, 2>(L, io, pl, sl2, r, s);
        }
    }
    switch (pl.waves) {
        case 8: return launch_step_bf16<64, 8>(L, io, pl, sl2, r, s);
        case 4: return launch_step_bf16<64, 4>(L, io, pl, sl2, r, s);
        default: return launch_step_bf16<64, 2>(L, io, pl, sl2, r, s);
    }
}

hipError_t launch_epilogue(const LayerView& L, const StepIO& io, double r, hipStream_t stream) {
    const int merge = !(L.bf16 && L.nsplit == 1);  // else the step kernel wrote the outputs
    const size_t shm = (size_t)L.S * (8 + 12) + (L.agg ? (size_t)L.hgrp * L.G * 16 : 0) +
                       (merge ? ((size_t)2 * L.nsplit * L.G + L.G) * 4 : 0);
    const dim3 grid((unsigned)(L.U / L.hgrp));
    const dim3 block(grid.x < 256 ? 1024 : 256);  // fewer workgroups than CUs: more threads each
    if (L.bf16)
        hipLaunchKernelGGL(k_epilogue<uint16_t>, grid, block, shm, stream, L, io, r, merge);
    else
        hipLaunchKernelGGL(k_epilogue<float>, grid, block, shm, stream, L, io, r, merge);
    return hipGetLastError();
}

}  // namespace raas
