// k_attention.hip -- grouped-query attention over the per-sequence KV cache.
//
// bf16 path (split-KV, MFMA).  One wave owns one work item: up to 16 query
// columns (query tokens x the q-heads of one kv-head) against one chunk of
// key positions of one KV slot.  Every K and V byte of the chunk is read
// once for all q-heads of the group.  A pair item serves the single decode
// tokens of two sequences that read the same shared prompt chunk (2 x group
// columns), so that chunk is read once for both.
//   scores   S^T[t][c] = K[t] . Q[c]     (A = 16 key rows, B = 16 columns)
//   output   O^T[d][c] += V^T[d][t] P^T[t][c]
// Key rows of the two 16-row score tiles of a 32-position step are permuted
// so that the lane holding column c and k-group q owns the scores of
// positions t0 + 8q .. t0 + 8q + 7; those eight probabilities are exactly
// the lane's B operand of the P.V product, and the matching A operand is one
// 16-byte load from the V cache's 8-position blocks.  No LDS, no transposes.
// Online softmax in the exp2 domain, fp32 state; the probabilities enter the
// P.V MFMA as a bf16 hi/lo pair, so they are not rounded to bf16.  A work
// item that covers all keys of its tokens writes the normalised output;
// otherwise it writes (max, sum, unnormalised output) partials that
// attn_combine merges in item order.  (Merging in the last-arriving wave
// would need device-scope fences, which on this multi-XCD part write back and
// invalidate the whole L2 and slow every co-running wave.)
//
// fp32 path: one workgroup per (row, q-head), plain VALU (tiny model only).
#include <hip/hip_ext.h>

#include "rl_device.h"
#include "rl_internal.h"

namespace rl {

// Zero the bf16 elements e >= nvalid of an 8-element vector (0 <= nvalid <= 8).
__device__ __forceinline__ u32x4 mask_tail8(u32x4 v, int nvalid) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int e0 = 2 * w;
        uint32_t keep = (e0 < nvalid ? 0x0000FFFFu : 0u) | (e0 + 1 < nvalid ? 0xFFFF0000u : 0u);
        v[w] &= keep;
    }
    return v;
}

// One 32-position step of the online-softmax attention of a wave's 16 query
// columns: scores of positions t0..t0+31 from the K rows (k0: tile 0, k1:
// tile 1), positions past min(hi - 1, limit) masked, running max / sum / output
// updated with the V blocks vf (positions >= hi zeroed).
template <int D>
__device__ __forceinline__ void attn_step(const u32x4 (&k0)[D / 32], const u32x4 (&k1)[D / 32],
                                          const u32x4 (&vf)[D / 16], const u32x4 (&qf)[D / 32], int t0, int hi,
                                          int limit, int kq, float scale_log2, float& m, float& l,
                                          f32x4 (&o)[D / 16]) {
    constexpr int KG = D / 32, DT = D / 16;
    const int pb = t0 + 8 * kq;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KG; ++j) {
        s0 = mfma16x16x32(as_bf16x8(k0[j]), as_bf16x8(qf[j]), s0);
        s1 = mfma16x16x32(as_bf16x8(k1[j]), as_bf16x8(qf[j]), s1);
    }
    // this lane now holds the scores of its column at positions pb + 0..7
    const int lim = min(hi - 1, limit);
    float sv[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        sv[e] = (pb + e <= lim) ? s0[e] * scale_log2 : -INFINITY;
        sv[4 + e] = (pb + 4 + e <= lim) ? s1[e] * scale_log2 : -INFINITY;
    }
    float mx = sv[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m, mx);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = exp2f(m - m_use);
    // probabilities as a bf16 pair hi + lo (hi = rne(p), lo = rne(p - hi)):
    // the P.V product then carries ~16 significant bits of p, so the only
    // storage rounding left is the one of the attention output
    float psum = 0.0f;
    uint32_t ph[4], pl[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const float p0 = exp2f(sv[2 * w] - m_use);
        const float p1 = exp2f(sv[2 * w + 1] - m_use);
        psum += p0 + p1;
        const uint16_t h0 = f32_to_bf16(p0), h1 = f32_to_bf16(p1);
        const uint16_t l0 = f32_to_bf16(p0 - bf16_to_f32(h0)), l1 = f32_to_bf16(p1 - bf16_to_f32(h1));
        ph[w] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
        pl[w] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
    }
    l = l * alpha + psum;
    m = m_new;
    const u32x4 pfh = {ph[0], ph[1], ph[2], ph[3]};
    const u32x4 pfl = {pl[0], pl[1], pl[2], pl[3]};
    const int nvalid = hi - pb;   // keys past the chunk end carry no data
#pragma unroll
    for (int i = 0; i < DT; ++i) {
        u32x4 v = nvalid < 8 ? mask_tail8(vf[i], nvalid < 0 ? 0 : nvalid) : vf[i];
        o[i] = o[i] * alpha;
        o[i] = mfma16x16x32(as_bf16x8(v), as_bf16x8(pfh), o[i]);
        o[i] = mfma16x16x32(as_bf16x8(v), as_bf16x8(pfl), o[i]);
    }
}

// 16-byte chunk permutation of K row r (of a 32-position step) in LDS:
// logical chunk c sits at c ^ kswz(r), which makes the fragment reads of one
// 16-lane group hit 16 different 16-byte bank groups.
template <int D>
__device__ __forceinline__ int kswz(int r) {
    return D == 128 ? ((r & 3) | ((r >> 1) & 12)) : (((r >> 1) & 1) | ((r >> 2) & 6));
}

__device__ __forceinline__ void lds_dma16(const void* g, uint8_t* lds_wave_base) {
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)(lds_wave_base), 16, 0, 0);
}

// The K rows and V blocks of positions t0..t0+31 of one (slot, kv-head) into
// an LDS step buffer (K [32][D] chunk-permuted, V [4][D][8]), spread over the
// kWaves waves of the workgroup: wave w moves KB w, w + kWaves, ... of each
// (waves past the step's KB count move none).  One global_load_lds per KB per
// lane.
template <int D, int kWaves>
__device__ __forceinline__ void step_dma(const uint16_t* kb, const uint16_t* vb, int t0, int wave, int lane,
                                         uint8_t* kl, uint8_t* vl) {
    constexpr int STEPB = 32 * D * 2;
    constexpr int NKB = STEPB / 1024;     // KB of K (and of V) per step
    constexpr int RPK = 1024 / (D * 2);   // K rows per KB
    constexpr int CPR = D / 8;            // 16-byte chunks per row
#pragma unroll
    for (int j = 0; j < (NKB + kWaves - 1) / kWaves; ++j) {
        const int kb_ = wave + kWaves * j;
        if (kb_ >= NKB) break;
        const int r = kb_ * RPK + lane / CPR;
        const int c = (lane % CPR) ^ kswz<D>(r);
        lds_dma16(kb + static_cast<size_t>(t0 + r) * D + 8 * c, kl + kb_ * 1024);
        lds_dma16(reinterpret_cast<const uint8_t*>(vb + static_cast<size_t>(t0) * D) + kb_ * 1024 + lane * 16,
                  vl + kb_ * 1024);
    }
}

// A wave's K / V fragments of one step from an LDS step buffer.
template <int D>
__device__ __forceinline__ void step_frags(const uint8_t* kl, const uint8_t* vl, int krow, int kq, int col,
                                           u32x4 (&k0)[D / 32], u32x4 (&k1)[D / 32], u32x4 (&vf)[D / 16]) {
#pragma unroll
    for (int j = 0; j < D / 32; ++j) {
        const int c = kq + 4 * j;
        k0[j] = *reinterpret_cast<const u32x4*>(kl + krow * (2 * D) + 16 * (c ^ kswz<D>(krow)));
        k1[j] = *reinterpret_cast<const u32x4*>(kl + (krow + 4) * (2 * D) + 16 * (c ^ kswz<D>(krow + 4)));
    }
#pragma unroll
    for (int i = 0; i < D / 16; ++i) vf[i] = *reinterpret_cast<const u32x4*>(vl + (kq * D + col + 16 * i) * 16);
}

// vmcnt(0) with expcnt and lgkmcnt left alone (gfx9 encoding)
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

// PAGED: the item's key range may cross pages, so each 32-position step
// looks its page up; otherwise the slot's block is fixed for the item.
template <int D, bool PAGED>
__global__ void __launch_bounds__(256, 2) attn_bf16_kernel(const AttnItem* __restrict__ items,
        int n_items, const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
        const uint16_t* __restrict__ vc, KvPages kp, int Hq, int Hkv, int layer,
        float scale_log2, uint16_t* __restrict__ out, float* __restrict__ part) {
    constexpr int KG = D / 32;   // 32-wide k groups of a head
    constexpr int DT = D / 16;   // 16-wide d tiles of the output
    constexpr int STEPB = 32 * D * 2;
    __shared__ __attribute__((aligned(1024))) uint8_t lds[2][2][STEPB];   // [buffer][K | V], shared-chunk units
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int item_id = blockIdx.x * 4 + wave;
    // a unit of four items over one shared prompt chunk (same slot and key
    // range; the host sets pad = 1 on its first item): every K/V step goes
    // through LDS once for the four waves
    const bool wg_lds = blockIdx.x * 4 + 3 < n_items && items[blockIdx.x * 4].pad == 1;
    if (item_id >= n_items) return;
    const int kvh = blockIdx.y;
    const int G = Hq / Hkv;
    const AttnItem it = items[item_id];

    const int col = lane & 15, kq = lane >> 4;
    const int ncols = it.nq * G;
    const bool cvalid = col < ncols;
    const int tau = cvalid ? col / G : 0;
    const int head = kvh * G + (cvalid ? col - tau * G : 0);
    const bool second = it.qrow_b >= 0 && tau == 1;   // second sequence of a pair item
    const int qrow = second ? it.qrow_b : it.qrow + tau;
    const int limit = cvalid ? it.pos0 + tau : -1;   // last key this column sees

    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 qf[KG];
    {
        const uint16_t* qp = q + (static_cast<size_t>(qrow) * Hq + head) * D + 8 * kq;
#pragma unroll
        for (int j = 0; j < KG; ++j) qf[j] = cvalid ? ld16(qp + 32 * j) : zero;
    }

    // K / V block of the step at position t0 (element pointers) and t0's
    // position inside it.  A paged item reads the table entry of its first
    // page here, right after the q loads, and each later entry one page
    // ahead (steps ascend 32 positions at a time, so they enter pages in
    // order).
    size_t base = 0;
    int base_page = 0, next_pid = 0;
    if (!PAGED) {
        base = kv_block(kp, layer, Hkv, it.slot, kvh);
    } else {
        base_page = it.kv_lo / kp.page;
        if (base_page < kp.maxp) base = kv_block(kp, layer, Hkv, kv_clamp(kp, kv_table(kp, it.slot, base_page)), kvh);
        if (base_page + 1 < kp.maxp) next_pid = kv_table(kp, it.slot, base_page + 1);
    }
    auto block_of = [&](int t0, const uint16_t** kbp, const uint16_t** vbp) {
        int lt = t0;
        if (PAGED) {
            const int j = t0 / kp.page;
            if (j != base_page) {
                const int pid = j == base_page + 1 ? next_pid : kv_table(kp, it.slot, j);
                base = kv_block(kp, layer, Hkv, kv_clamp(kp, pid), kvh);
                base_page = j;
                next_pid = j + 1 < kp.maxp ? kv_table(kp, it.slot, j + 1) : 0;
            }
            lt = t0 - j * kp.page;
        }
        *kbp = kc + base;
        *vbp = vc + base;
        return lt;
    };

    float m = -INFINITY, l = 0.0f;
    f32x4 o[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int hi = it.kv_hi;
    // key row r of score tile 0 is position t0 + 8(r/4) + r%4; tile 1 adds 4
    const int krow = 8 * (col >> 2) + (col & 3);
    // K rows and V blocks of one 32-position step, loaded and then used (the
    // waves resident on the chip keep HBM busy without a per-wave prefetch)
    u32x4 k0[KG], k1[KG], vf[DT];
    auto load_step = [&](int t0, u32x4 (&a0)[KG], u32x4 (&a1)[KG], u32x4 (&vv)[DT]) {
        const uint16_t *kb, *vb;
        const int lt = block_of(t0, &kb, &vb);
        const uint16_t* kp0 = kb + static_cast<size_t>(lt + krow) * D + 8 * kq;
        const uint16_t* kp1 = kp0 + 4 * D;
#pragma unroll
        for (int j = 0; j < KG; ++j) {
            a0[j] = ld16(kp0 + 32 * j);
            a1[j] = ld16(kp1 + 32 * j);
        }
        const uint16_t* vp = vb + (static_cast<size_t>((lt + 8 * kq) >> 3) * D + col) * 8;
#pragma unroll
        for (int i = 0; i < DT; ++i) vv[i] = ld16(vp + 16 * 8 * i);
    };
    auto dma_step = [&](int t0, int buf) {
        const uint16_t *kb, *vb;
        const int lt = block_of(t0, &kb, &vb);
        step_dma<D, 4>(kb, vb, lt, wave, lane, lds[buf][0], lds[buf][1]);
    };
    if (wg_lds) {
        const int nsteps = (hi - it.kv_lo + 31) / 32;
        if (nsteps > 0) dma_step(it.kv_lo, 0);
        for (int s = 0; s < nsteps; ++s) {
            wait_vm0();        // this wave's DMAs (and q loads) landed
            __syncthreads();   // every wave's part of step s is in LDS; step s-1 retired
            if (s + 1 < nsteps) dma_step(it.kv_lo + 32 * (s + 1), (s + 1) & 1);
            step_frags<D>(lds[s & 1][0], lds[s & 1][1], krow, kq, col, k0, k1, vf);
            attn_step<D>(k0, k1, vf, qf, it.kv_lo + 32 * s, hi, limit, kq, scale_log2, m, l, o);
        }
    } else {
        for (int t0 = it.kv_lo; t0 < hi; t0 += 32) {
            load_step(t0, k0, k1, vf);
            attn_step<D>(k0, k1, vf, qf, t0, hi, limit, kq, scale_log2, m, l, o);
        }
    }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);

    // lane holds O^T[d = 16 i + 4 kq + e][col]
    if (it.part < 0) {
        if (!cvalid) return;
        const float inv = 1.0f / l;
        uint16_t* op = out + (static_cast<size_t>(qrow) * Hq + head) * D + 4 * kq;
#pragma unroll
        for (int i = 0; i < DT; ++i) {
            const uint32_t w0 = static_cast<uint32_t>(f32_to_bf16(o[i][0] * inv)) |
                                (static_cast<uint32_t>(f32_to_bf16(o[i][1] * inv)) << 16);
            const uint32_t w1 = static_cast<uint32_t>(f32_to_bf16(o[i][2] * inv)) |
                                (static_cast<uint32_t>(f32_to_bf16(o[i][3] * inv)) << 16);
            *reinterpret_cast<uint2*>(op + 16 * i) = make_uint2(w0, w1);
        }
        return;
    }
    // split block: (m, l, unnormalised o) partials, merged by attn_combine
    if (!cvalid) return;
    // a pair item's second sequence owns its own partial slot (columns from 0)
    const int pidx = second ? it.part_b : it.part;
    const int pcol = second ? col - G : col;
    float* pp = part + ((static_cast<size_t>(pidx) * Hkv + kvh) * 16 + pcol) * (D + 2);
#pragma unroll
    for (int i = 0; i < DT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) pp[16 * i + 4 * kq + e] = o[i][e];
    if (kq == 0) {
        pp[D] = m;
        pp[D + 1] = l;
    }
}

hipError_t launch_attention_bf16(const AttnItem* items, int n_items, const void* q,
                                 const void* kc, const void* vc, const KvPages& kp, int Hq, int Hkv,
                                 int D, int layer, void* out, float* part,
                                 hipStream_t s, hipEvent_t ev_start, hipEvent_t ev_stop) {
    if (n_items <= 0) return hipSuccess;
    const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    dim3 grid((n_items + 3) / 4, Hkv), block(256);
    auto go = [&](auto kern) {
        if (ev_start || ev_stop)
            hipExtLaunchKernelGGL(kern, grid, block, 0, s, ev_start, ev_stop, 0, items, n_items,
                                  static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(kc),
                                  static_cast<const uint16_t*>(vc), kp, Hq, Hkv, layer, scale_log2,
                                  static_cast<uint16_t*>(out), part);
        else
            hipLaunchKernelGGL(kern, grid, block, 0, s, items, n_items, static_cast<const uint16_t*>(q),
                               static_cast<const uint16_t*>(kc), static_cast<const uint16_t*>(vc), kp, Hq,
                               Hkv, layer, scale_log2, static_cast<uint16_t*>(out), part);
    };
    if (kp.table) {
        if (D == 128) go(attn_bf16_kernel<128, true>); else go(attn_bf16_kernel<64, true>);
    } else {
        if (D == 128) go(attn_bf16_kernel<128, false>); else go(attn_bf16_kernel<64, false>);
    }
    return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Prefill / scoring attention: a workgroup of kPrefillWaves waves shares each
// K/V step through LDS.  Per 32-position step the workgroup DMAs the step's K rows
// ([32][D], 16-byte chunks permuted by row so that the fragment reads below
// are free of bank conflicts) and its four V blocks ([4][D][8], contiguous in
// the cache) into one of two LDS buffers with global_load_lds; every wave
// then runs the decode kernel's MFMA step on its own 16 query columns from
// LDS.  The next step's DMA is issued right after the barrier that retires
// the previous step, so it overlaps the current step's math.
// ---------------------------------------------------------------------------

template <int D>
__global__ void __launch_bounds__(64 * kPrefillWaves) attn_prefill_kernel(const PrefillTile* __restrict__ tiles,
        const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
        KvPages kp, int Hq, int Hkv, int layer, float scale_log2, uint16_t* __restrict__ out) {
    constexpr int KG = D / 32, DT = D / 16;
    constexpr int STEPB = 32 * D * 2;               // bytes of K (and of V) per 32-position step
    static_assert(STEPB % 1024 == 0, "whole 1 KB DMA instructions per step");
    __shared__ __attribute__((aligned(1024))) uint8_t lds[2][2][STEPB];   // [buffer][K | V]

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int kvh = blockIdx.y;
    const int G = Hq / Hkv;
    const int tq = 16 / G;
    const PrefillTile tl = tiles[blockIdx.x];
    const int tok0 = wave * tq;
    const int nq = max(0, min(tq, tl.ntok - tok0));
    const int col = lane & 15, kq = lane >> 4;
    const bool cvalid = col < nq * G;
    const int tau = cvalid ? col / G : 0;
    const int head = kvh * G + (cvalid ? col - tau * G : 0);
    const int qrow = cvalid ? tl.qrow0 + tok0 + tau : tl.qrow0;
    const int limit = cvalid ? tl.pos0 + tok0 + tau : -1;
    const int hi = tl.pos0 + tl.ntok;               // keys [0, hi)
    const int wave_last = tl.pos0 + tok0 + nq - 1;  // last key any column of this wave sees
    const int nsteps = (hi + 31) / 32;

    // the K/V of the step at position t0: its page's blocks and t0 inside the page
    auto dma_step = [&](int t0, int buf) {
        int lt;
        const size_t b = kv_block(kp, layer, Hkv, kv_page(kp, tl.slot, t0, &lt), kvh);
        step_dma<D, kPrefillWaves>(kc + b, vc + b, lt, wave, lane, lds[buf][0], lds[buf][1]);
    };

    const u32x4 zero = {0u, 0u, 0u, 0u};
    u32x4 qf[KG];
    {
        const uint16_t* qp = q + (static_cast<size_t>(qrow) * Hq + head) * D + 8 * kq;
#pragma unroll
        for (int j = 0; j < KG; ++j) qf[j] = cvalid ? ld16(qp + 32 * j) : zero;
    }
    float m = -INFINITY, l = 0.0f;
    f32x4 o[DT];
#pragma unroll
    for (int i = 0; i < DT; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int krow = 8 * (col >> 2) + (col & 3);

    if (nsteps > 0) dma_step(0, 0);
    for (int s = 0; s < nsteps; ++s) {
        wait_vm0();        // this wave's DMAs (and q loads) landed
        __syncthreads();   // every wave's part of step s is in LDS; step s-1 retired
        if (s + 1 < nsteps) dma_step(32 * (s + 1), (s + 1) & 1);
        const int t0 = 32 * s;
        if (nq == 0 || t0 > wave_last) continue;       // wave-uniform: nothing of this step is visible
        u32x4 k0[KG], k1[KG], vf[DT];
        step_frags<D>(lds[s & 1][0], lds[s & 1][1], krow, kq, col, k0, k1, vf);
        attn_step<D>(k0, k1, vf, qf, t0, hi, limit, kq, scale_log2, m, l, o);
    }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    if (!cvalid) return;
    const float inv = 1.0f / l;
    uint16_t* op = out + (static_cast<size_t>(qrow) * Hq + head) * D + 4 * kq;
#pragma unroll
    for (int i = 0; i < DT; ++i) {
        const uint32_t w0 = static_cast<uint32_t>(f32_to_bf16(o[i][0] * inv)) |
                            (static_cast<uint32_t>(f32_to_bf16(o[i][1] * inv)) << 16);
        const uint32_t w1 = static_cast<uint32_t>(f32_to_bf16(o[i][2] * inv)) |
                            (static_cast<uint32_t>(f32_to_bf16(o[i][3] * inv)) << 16);
        *reinterpret_cast<uint2*>(op + 16 * i) = make_uint2(w0, w1);
    }
}

hipError_t launch_attention_prefill(const PrefillTile* tiles, int n_tiles, const void* q, const void* kc,
                                    const void* vc, const KvPages& kp, int Hq, int Hkv, int D, int layer,
                                    void* out, hipStream_t s) {
    if (n_tiles <= 0) return hipSuccess;
    const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    dim3 grid(n_tiles, Hkv), block(64 * kPrefillWaves);
    if (D == 128)
        hipLaunchKernelGGL(attn_prefill_kernel<128>, grid, block, 0, s, tiles, static_cast<const uint16_t*>(q),
                           static_cast<const uint16_t*>(kc), static_cast<const uint16_t*>(vc), kp, Hq, Hkv,
                           layer, scale_log2, static_cast<uint16_t*>(out));
    else
        hipLaunchKernelGGL(attn_prefill_kernel<64>, grid, block, 0, s, tiles, static_cast<const uint16_t*>(q),
                           static_cast<const uint16_t*>(kc), static_cast<const uint16_t*>(vc), kp, Hq, Hkv,
                           layer, scale_log2, static_cast<uint16_t*>(out));
    return hipGetLastError();
}

// Merge the split partials of one query block and q-head: one workgroup per
// (split block, q-head), one thread per d, the block's tokens in turn.  Lane
// j of each wave loads item j's (m, l) (at most 64 items), the token's max
// comes from a wave reduction, and each thread sums its own column of the
// partial outputs in item order, 8 loads in flight at a time, reading the
// items' (m, l) from their lanes.  Weights 2^(m_j - M).
template <int D>
__global__ void __launch_bounds__(D) attn_combine_kernel(const int32_t* __restrict__ blocks,
        const AttnItem* __restrict__ items, const float* __restrict__ part, int Hq, int Hkv,
        uint16_t* __restrict__ out) {
    static_assert(kMaxCombine <= 64, "one item per lane");
    const AttnItem it = items[blocks[blockIdx.x]];
    const int h = blockIdx.y;
    const int G = Hq / Hkv;
    const int kvh = h / G, g = h - kvh * G;
    const int np = it.nparts;
    const int d = threadIdx.x, lane = threadIdx.x & 63;
    const size_t pstride = static_cast<size_t>(Hkv) * 16 * (D + 2);
    const float* pb0 = part + (static_cast<size_t>(it.part0) * Hkv + kvh) * 16 * (D + 2);
    auto lane_f = [](float v, int src) {
        return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), src));
    };
    for (int t = 0; t < it.nq; ++t) {
        const float* pc = pb0 + static_cast<size_t>(t * G + g) * (D + 2);
        const float mv = lane < np ? pc[lane * pstride + D] : -INFINITY;
        const float lv = lane < np ? pc[lane * pstride + D + 1] : 0.0f;
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (u < np) v[u] = pc[u * pstride + d];
        float M = mv;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off, 64));
        float acc = 0.0f, L = 0.0f;
        for (int j = 0; j < np; j += 8) {
            if (j > 0) {
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (j + u < np) v[u] = pc[(j + u) * pstride + d];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                if (j + u < np) {
                    const float w = exp2f(lane_f(mv, j + u) - M);
                    L += w * lane_f(lv, j + u);
                    acc += w * v[u];
                }
            }
        }
        out[(static_cast<size_t>(it.qrow + t) * Hq + h) * D + d] = f32_to_bf16(acc / L);
    }
}

hipError_t launch_attn_combine(const int32_t* blocks, int n_blocks, const AttnItem* items, const float* part,
                               int Hq, int Hkv, int D, void* out, hipStream_t s) {
    if (n_blocks <= 0) return hipSuccess;
    dim3 grid(n_blocks, Hq), block(D);
    if (D == 128)
        hipLaunchKernelGGL(attn_combine_kernel<128>, grid, block, 0, s, blocks, items, part, Hq, Hkv,
                           static_cast<uint16_t*>(out));
    else
        hipLaunchKernelGGL(attn_combine_kernel<64>, grid, block, 0, s, blocks, items, part, Hq, Hkv,
                           static_cast<uint16_t*>(out));
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// fp32: one 64-lane workgroup per (row, q-head); keys 0..pos of the row's slot.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(64) attn_f32_kernel(const int32_t* __restrict__ row_slot,
        const int32_t* __restrict__ row_pos, const float* __restrict__ q,
        const float* __restrict__ kc, const float* __restrict__ vc, KvPages kp, int Hq, int Hkv, int D,
        int layer, float* __restrict__ out) {
    __shared__ float qs[128];
    __shared__ float ps[64];
    const int r = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
    const int G = Hq / Hkv, kvh = h / G;
    const int pos = row_pos[r], slot = row_slot[r];
    const float* qr = q + (static_cast<size_t>(r) * Hq + h) * D;
    for (int i = lane; i < D; i += 64) qs[i] = qr[i];
    __syncthreads();
    // K row and V block start of position t (its page's block, t inside it)
    auto krow_of = [&](int t) {
        int lt;
        const size_t b = kv_block(kp, layer, Hkv, kv_page(kp, slot, t, &lt), kvh);
        return kc + b + static_cast<size_t>(lt) * D;
    };
    auto vblk_of = [&](int t) {
        int lt;
        const size_t b = kv_block(kp, layer, Hkv, kv_page(kp, slot, t, &lt), kvh);
        return vc + b + static_cast<size_t>(lt >> 3) * D * 8 + (lt & 7);
    };
    const float scale = 1.0f / sqrtf(static_cast<float>(D));
    float m = -INFINITY, l = 0.0f;
    float acc0 = 0.0f, acc1 = 0.0f;   // d = lane, lane + 64
    for (int t0 = 0; t0 <= pos; t0 += 64) {
        const int t = t0 + lane;
        float s = -INFINITY;
        if (t <= pos) {
            const float* kr = krow_of(t);
            float d = 0.0f;
            for (int i = 0; i < D; ++i) d = fmaf(qs[i], kr[i], d);
            s = d * scale;
        }
        const float mx = wave_max(s);
        const float m_new = fmaxf(m, mx);
        const float alpha = expf(m - m_new);
        const float p = t <= pos ? expf(s - m_new) : 0.0f;
        l = l * alpha + wave_sum(p);
        m = m_new;
        ps[lane] = p;
        __syncthreads();
        acc0 *= alpha;
        acc1 *= alpha;
        const int nt = min(64, pos + 1 - t0);
        for (int tt = 0; tt < nt; ++tt) {
            const float* vblk = vblk_of(t0 + tt);
            if (lane < D) acc0 = fmaf(ps[tt], vblk[static_cast<size_t>(lane) * 8], acc0);
            if (lane + 64 < D) acc1 = fmaf(ps[tt], vblk[static_cast<size_t>(lane + 64) * 8], acc1);
        }
        __syncthreads();
    }
    float* orow = out + (static_cast<size_t>(r) * Hq + h) * D;
    if (lane < D) orow[lane] = acc0 / l;
    if (lane + 64 < D) orow[lane + 64] = acc1 / l;
}

hipError_t launch_attention_f32(int n_rows, const int32_t* row_slot, const int32_t* row_pos,
                                const float* q, const float* kc, const float* vc, const KvPages& kp,
                                int Hq, int Hkv, int D, int layer, float* out,
                                hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(attn_f32_kernel, dim3(n_rows, Hq), dim3(64), 0, s, row_slot, row_pos, q, kc,
                       vc, kp, Hq, Hkv, D, layer, out);
    return hipGetLastError();
}

}  // namespace rl
