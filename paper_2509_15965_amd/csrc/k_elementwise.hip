// k_elementwise.hip -- embedding gather, RMSNorm, RoPE + KV append, copy probe.
#include "rl_device.h"
#include "rl_internal.h"

namespace rl {

// x[r][:] = fp32(row of the embedding table or of the caller's rows), and
// optionally h[r][:] = storage(x / sqrt(mean(x^2) + eps) * g) (the first
// layer's attention norm).  tok >= 0 selects table row tok (< V); tok < 0
// selects rows[-tok-1] (< n_rows); anything else embeds as zeros.
template <typename T>
__global__ void __launch_bounds__(256) embed_kernel(const int32_t* __restrict__ tok,
        const T* __restrict__ table, int V, const T* __restrict__ rows, int n_rows, int H,
        float* __restrict__ x, const T* __restrict__ g, float eps, T* __restrict__ h) {
    __shared__ float red[4];
    const int r = blockIdx.x;
    const int t = tok[r];
    const T* src = nullptr;
    if (t >= 0 && t < V) src = table + static_cast<size_t>(t) * H;
    else if (t < 0 && rows != nullptr && -(t + 1) < n_rows) src = rows + static_cast<size_t>(-(t + 1)) * H;
    float* dst = x + static_cast<size_t>(r) * H;
    float ss = 0.0f;
    bool vec = false;
    if constexpr (sizeof(T) == 2)
        vec = H % 8 == 0 && H <= 8 * 4 * 256 && (reinterpret_cast<uintptr_t>(src) & 15) == 0;
    if (vec) {
        // 16-byte loads, every one of the thread's loads in flight at once
        constexpr int P = 4;
        u32x4 raw[P];
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const int c = threadIdx.x + 256 * j;
            raw[j] = src && 8 * c < H ? ld16(src + 8 * c) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < P; ++j) {
            const int c = threadIdx.x + 256 * j;
            if (8 * c >= H) continue;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float v = bf16_to_f32(static_cast<uint16_t>(raw[j][e >> 1] >> (16 * (e & 1))));
                dst[8 * c + e] = v;
                ss = fmaf(v, v, ss);
            }
        }
    } else {
        for (int i = threadIdx.x; i < H; i += blockDim.x) {
            const float v = src ? Elem<T>::load(src, i) : 0.0f;
            dst[i] = v;
            ss = fmaf(v, v, ss);
        }
    }
    if (h == nullptr) return;
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = red[0] + red[1] + red[2] + red[3];
    const float rs = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
    T* hr = h + static_cast<size_t>(r) * H;
    for (int i = threadIdx.x; i < H; i += blockDim.x) Elem<T>::store(hr, i, dst[i] * rs * Elem<T>::load(g, i));
}

hipError_t launch_embed(int dt, const int32_t* tok, int n, const void* table, int V,
                        const void* rows, int n_rows, int H, float* x, const void* g, float eps, void* h,
                        hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (dt == DT_BF16)
        hipLaunchKernelGGL(embed_kernel<uint16_t>, dim3(n), dim3(256), 0, s, tok,
                           static_cast<const uint16_t*>(table), V,
                           static_cast<const uint16_t*>(rows), n_rows, H, x,
                           static_cast<const uint16_t*>(g), eps, static_cast<uint16_t*>(h));
    else
        hipLaunchKernelGGL(embed_kernel<float>, dim3(n), dim3(256), 0, s, tok,
                           static_cast<const float*>(table), V, static_cast<const float*>(rows),
                           n_rows, H, x, static_cast<const float*>(g), eps, static_cast<float*>(h));
    return hipGetLastError();
}

// out[o][:] = storage( x[row] / sqrt(mean(x[row]^2) + eps) * g ), row = sel ? sel[o] : o.
// fp32 statistics; one workgroup per row.
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_kernel(const float* __restrict__ x,
        const int32_t* __restrict__ sel, int H, const T* __restrict__ g, float eps,
        T* __restrict__ out) {
    __shared__ float red[4];
    const int o = blockIdx.x;
    const int row = sel ? sel[o] : o;
    const float* xr = x + static_cast<size_t>(row) * H;
    float ss = 0.0f;
    for (int i = threadIdx.x; i < H; i += 256) {
        float v = xr[i];
        ss = fmaf(v, v, ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = red[0] + red[1] + red[2] + red[3];
    const float r = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
    T* orow = out + static_cast<size_t>(o) * H;
    for (int i = threadIdx.x; i < H; i += 256)
        Elem<T>::store(orow, i, xr[i] * r * Elem<T>::load(g, i));
}

// The same norm with 16-byte accesses (H a multiple of 4): the row is read
// once into registers (PER float4 per thread) and reused for the output.
template <typename T, int PER>
__global__ void __launch_bounds__(256) rmsnorm4_kernel(const float* __restrict__ x,
        const int32_t* __restrict__ sel, int H, const T* __restrict__ g, float eps,
        T* __restrict__ out) {
    __shared__ float red[4];
    const int o = blockIdx.x;
    const int row = sel ? sel[o] : o;
    const f32x4* xr = reinterpret_cast<const f32x4*>(x + static_cast<size_t>(row) * H);
    const int H4 = H / 4;
    f32x4 v[PER];
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int c = threadIdx.x + 256 * j;
        v[j] = c < H4 ? xr[c] : f32x4{0.f, 0.f, 0.f, 0.f};
        ss = fmaf(v[j][0], v[j][0], ss);
        ss = fmaf(v[j][1], v[j][1], ss);
        ss = fmaf(v[j][2], v[j][2], ss);
        ss = fmaf(v[j][3], v[j][3], ss);
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = red[0] + red[1] + red[2] + red[3];
    const float r = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
    T* orow = out + static_cast<size_t>(o) * H;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int c = threadIdx.x + 256 * j;
        if (c < H4) {
#pragma unroll
            for (int e = 0; e < 4; ++e) Elem<T>::store(orow, 4 * c + e, v[j][e] * r * Elem<T>::load(g, 4 * c + e));
        }
    }
}

hipError_t launch_rmsnorm(int dt, const float* x, const int32_t* sel, int n, int H,
                          const void* g, float eps, void* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int per = (H / 4 + 255) / 256;
    if (H % 4 == 0 && per <= 8) {
#define RL_N4(P)                                                                                          \
        do {                                                                                              \
            if (dt == DT_BF16)                                                                            \
                hipLaunchKernelGGL((rmsnorm4_kernel<uint16_t, P>), dim3(n), dim3(256), 0, s, x, sel, H,  \
                                   static_cast<const uint16_t*>(g), eps, static_cast<uint16_t*>(out));   \
            else                                                                                          \
                hipLaunchKernelGGL((rmsnorm4_kernel<float, P>), dim3(n), dim3(256), 0, s, x, sel, H,     \
                                   static_cast<const float*>(g), eps, static_cast<float*>(out));         \
        } while (0)
        if (per <= 2) RL_N4(2);
        else if (per <= 4) RL_N4(4);
        else RL_N4(8);
#undef RL_N4
        return hipGetLastError();
    }
    if (dt == DT_BF16)
        hipLaunchKernelGGL(rmsnorm_kernel<uint16_t>, dim3(n), dim3(256), 0, s, x, sel, H,
                           static_cast<const uint16_t*>(g), eps, static_cast<uint16_t*>(out));
    else
        hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(n), dim3(256), 0, s, x, sel, H,
                           static_cast<const float*>(g), eps, static_cast<float*>(out));
    return hipGetLastError();
}

// Split-K sum + residual + RMSNorm of one row per workgroup (H a multiple of 4):
//   x[r] += sum_{z < splits} part[z][r]   (in order z = 0, 1, ...)
//   out[r] = storage(x[r] / sqrt(mean(x[r]^2) + eps) * g)
// Each thread owns PER float4 of the row; the slices are loaded four at a
// time (every load of a group in flight together) and added in order, so the
// result equals the wide reduction followed by the norm.
template <typename T, int PER>
__global__ void __launch_bounds__(256) resid_norm4_kernel(const float* __restrict__ part, int splits,
        size_t slice, float* __restrict__ x, int H, const T* __restrict__ g, float eps, T* __restrict__ out) {
    __shared__ float red[4];
    const int r = blockIdx.x;
    const int H4 = H / 4;
    f32x4* xr = reinterpret_cast<f32x4*>(x + static_cast<size_t>(r) * H);
    const f32x4* pr = reinterpret_cast<const f32x4*>(part + static_cast<size_t>(r) * H);
    const size_t sl4 = slice / 4;
    f32x4 v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) v[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    int z = 0;
    for (; z + 4 <= splits; z += 4) {
        f32x4 t[4][PER];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < PER; ++j) {
                const int c = threadIdx.x + 256 * j;
                t[u][j] = c < H4 ? pr[(z + u) * sl4 + c] : f32x4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < PER; ++j) v[j] += t[u][j];
    }
    for (; z < splits; ++z)
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int c = threadIdx.x + 256 * j;
            if (c < H4) v[j] += pr[z * sl4 + c];
        }
    float ss = 0.0f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int c = threadIdx.x + 256 * j;
        if (c < H4) {
            const f32x4 nv = xr[c] + v[j];
            xr[c] = nv;
            v[j] = nv;
            ss = fmaf(nv[0], nv[0], ss);
            ss = fmaf(nv[1], nv[1], ss);
            ss = fmaf(nv[2], nv[2], ss);
            ss = fmaf(nv[3], nv[3], ss);
        }
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    ss = red[0] + red[1] + red[2] + red[3];
    const float rs = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
    T* orow = out + static_cast<size_t>(r) * H;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int c = threadIdx.x + 256 * j;
        if (c < H4) {
#pragma unroll
            for (int e = 0; e < 4; ++e) Elem<T>::store(orow, 4 * c + e, v[j][e] * rs * Elem<T>::load(g, 4 * c + e));
        }
    }
}

// The same pass with one float4 of the row per thread (H <= 4096, up to
// 1024 threads): every slice's load of a group of eight is in flight at
// once, so a row costs one or two memory round trips -- for batches too
// small to hide the latency of the grouped loads above.  Same order of
// additions; the sum of squares is reduced over the workgroup's waves.
template <typename T>
__global__ void __launch_bounds__(1024) resid_norm_wide_kernel(const float* __restrict__ part, int splits,
        size_t slice, float* __restrict__ x, int H, const T* __restrict__ g, float eps, T* __restrict__ out) {
    __shared__ float red[16];
    const int r = blockIdx.x, c = threadIdx.x;
    const int H4 = H / 4;
    const bool on = c < H4;
    f32x4* xr = reinterpret_cast<f32x4*>(x + static_cast<size_t>(r) * H);
    const f32x4* pr = reinterpret_cast<const f32x4*>(part + static_cast<size_t>(r) * H);
    const size_t sl4 = slice / 4;
    f32x4 v{0.f, 0.f, 0.f, 0.f};
    for (int z = 0; z < splits; z += 8) {
        f32x4 t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            t[u] = on && z + u < splits ? pr[(z + u) * sl4 + c] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (z + u < splits) v += t[u];
    }
    float ss = 0.0f;
    if (on) {
        v = xr[c] + v;
        xr[c] = v;
        ss = fmaf(v[0], v[0], ss);
        ss = fmaf(v[1], v[1], ss);
        ss = fmaf(v[2], v[2], ss);
        ss = fmaf(v[3], v[3], ss);
    }
    ss = wave_sum(ss);
    const int nw = (blockDim.x + 63) >> 6;
    if ((c & 63) == 0) red[c >> 6] = ss;
    __syncthreads();
    ss = 0.0f;
    for (int w = 0; w < nw; ++w) ss += red[w];
    const float rs = 1.0f / sqrtf(ss / static_cast<float>(H) + eps);
    if (on) {
        T* orow = out + static_cast<size_t>(r) * H;
#pragma unroll
        for (int e = 0; e < 4; ++e) Elem<T>::store(orow, 4 * c + e, v[e] * rs * Elem<T>::load(g, 4 * c + e));
    }
}

hipError_t launch_resid_norm(int dt, const float* part, int splits, float* x, int n, int H, const void* g,
                             float eps, void* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (H % 4 == 0 && H / 4 <= 1024) {
        const size_t slice = static_cast<size_t>(n) * H;
        const int threads = (H / 4 + 63) / 64 * 64;
        if (dt == DT_BF16)
            hipLaunchKernelGGL(resid_norm_wide_kernel<uint16_t>, dim3(n), dim3(threads), 0, s, part, splits, slice,
                               x, H, static_cast<const uint16_t*>(g), eps, static_cast<uint16_t*>(out));
        else
            hipLaunchKernelGGL(resid_norm_wide_kernel<float>, dim3(n), dim3(threads), 0, s, part, splits, slice,
                               x, H, static_cast<const float*>(g), eps, static_cast<float*>(out));
        return hipGetLastError();
    }
    const int per = (H / 4 + 255) / 256;
    if (H % 4 != 0 || per > 8) return hipErrorInvalidValue;
    const size_t slice = static_cast<size_t>(n) * H;
#define RL_RN(P)                                                                                            \
    do {                                                                                                    \
        if (dt == DT_BF16)                                                                                  \
            hipLaunchKernelGGL((resid_norm4_kernel<uint16_t, P>), dim3(n), dim3(256), 0, s, part, splits,  \
                               slice, x, H, static_cast<const uint16_t*>(g), eps, static_cast<uint16_t*>(out)); \
        else                                                                                                \
            hipLaunchKernelGGL((resid_norm4_kernel<float, P>), dim3(n), dim3(256), 0, s, part, splits,     \
                               slice, x, H, static_cast<const float*>(g), eps, static_cast<float*>(out));   \
    } while (0)
    if (per <= 2) RL_RN(2);
    else if (per <= 4) RL_RN(4);
    else RL_RN(8);
#undef RL_RN
    return hipGetLastError();
}

// Rotate-half RoPE on q and k (pairs i, i + D/2 rotated by the angle of the
// row's position at frequency i), storage rounding, and the KV append.  One
// thread per (row, head of q|k|v, pair i): it reads elements i and i + D/2 of
// the projection -- the sum, in split order, of `splits` fp32 split-K slices
// when the projection was split (no separate reduction pass) -- and writes q
// or the K / V cache entries of every destination slot (a negative row_dst
// entry names a single slot directly).
// cs: cos table [cap][D/2] followed by the sin table [cap][D/2].
// K cache element (l, s, h, t, i): (((l*S + s)*Hkv + h)*cap + t)*D + i.
// V cache element: ((((l*S + s)*Hkv + h)*(cap/8) + t/8)*D + i)*8 + t%8.
template <typename T>
__global__ void __launch_bounds__(256) rope_append_kernel(const float* __restrict__ qkv, int splits,
        size_t slice, int n_rows, const int32_t* __restrict__ row_pos, const int32_t* __restrict__ row_dst,
        int n_dst, const int32_t* __restrict__ dst_slots, const float* __restrict__ cs, int cs_stride, int Hq,
        int Hkv, int D, KvPages kp, int layer, T* __restrict__ q_out, T* __restrict__ kc,
        T* __restrict__ vc) {
    const int half = D / 2;
    const int nh = Hq + 2 * Hkv;
    const size_t gid = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (gid >= static_cast<size_t>(n_rows) * nh * half) return;
    const int i = static_cast<int>(gid % half);
    const int h = static_cast<int>((gid / half) % nh);
    const int r = static_cast<int>(gid / (static_cast<size_t>(half) * nh));
    const int nqkv = nh * D;
    const float* src = qkv + static_cast<size_t>(r) * nqkv + h * D + i;
    float a = src[0], b = src[half];
    for (int z = 1; z < splits; ++z) {
        a += src[z * slice];
        b += src[z * slice + half];
    }
    const int pos = row_pos[r];
    if (h < Hq + Hkv) {
        const float c = cs[static_cast<size_t>(pos) * half + i];
        const float sn = cs[static_cast<size_t>(cs_stride) + static_cast<size_t>(pos) * half + i];
        const float x0 = a * c - b * sn, x1 = b * c + a * sn;
        if (h < Hq) {
            T* qo = q_out + (static_cast<size_t>(r) * Hq + h) * D;
            Elem<T>::store(qo, i, x0);
            Elem<T>::store(qo, i + half, x1);
            return;
        }
        const int d0 = row_dst[r];
        const int nd = d0 < 0 ? 1 : n_dst;
        for (int g = 0; g < nd; ++g) {
            const int slot = d0 < 0 ? -(d0 + 1) : dst_slots[d0 + g];
            int lp;
            const int pid = kv_page(kp, slot, pos, &lp);
            T* kr = kc + kv_block(kp, layer, Hkv, pid, h - Hq) + static_cast<size_t>(lp) * D;
            Elem<T>::store(kr, i, x0);
            Elem<T>::store(kr, i + half, x1);
        }
        return;
    }
    const int d0 = row_dst[r];
    const int nd = d0 < 0 ? 1 : n_dst;
    for (int g = 0; g < nd; ++g) {
        const int slot = d0 < 0 ? -(d0 + 1) : dst_slots[d0 + g];
        int lp;
        const int pid = kv_page(kp, slot, pos, &lp);
        T* vb = vc + kv_block(kp, layer, Hkv, pid, h - Hq - Hkv);
        Elem<T>::store(vb, (static_cast<size_t>(lp >> 3) * D + i) * 8 + (lp & 7), a);
        Elem<T>::store(vb, (static_cast<size_t>(lp >> 3) * D + i + half) * 8 + (lp & 7), b);
    }
}

hipError_t launch_rope_append(int dt, const float* qkv, int splits, int n_rows, const int32_t* row_pos,
                              const int32_t* row_dst, int n_dst, const int32_t* dst_slots,
                              const float* cs, int cs_stride, int Hq, int Hkv, int D,
                              const KvPages& kp, int layer,
                              void* q_out, void* kc, void* vc, hipStream_t s) {
    if (n_rows <= 0) return hipSuccess;
    const size_t threads = static_cast<size_t>(n_rows) * (Hq + 2 * Hkv) * (D / 2);
    const size_t slice = static_cast<size_t>(n_rows) * (Hq + 2 * Hkv) * D;
    const dim3 grid(static_cast<unsigned>((threads + 255) / 256)), block(256);
    const int sp = splits < 1 ? 1 : splits;
    if (dt == DT_BF16)
        hipLaunchKernelGGL(rope_append_kernel<uint16_t>, grid, block, 0, s, qkv, sp, slice, n_rows, row_pos, row_dst,
                           n_dst, dst_slots, cs, cs_stride, Hq, Hkv, D, kp, layer,
                           static_cast<uint16_t*>(q_out), static_cast<uint16_t*>(kc), static_cast<uint16_t*>(vc));
    else
        hipLaunchKernelGGL(rope_append_kernel<float>, grid, block, 0, s, qkv, sp, slice, n_rows, row_pos, row_dst,
                           n_dst, dst_slots, cs, cs_stride, Hq, Hkv, D, kp, layer,
                           static_cast<float*>(q_out), static_cast<float*>(kc), static_cast<float*>(vc));
    return hipGetLastError();
}

// Live K/V of slots <-> a packed staging buffer (dir 0: pool -> stage, dir 1:
// stage -> pool).  One workgroup per (slot i, layer * Hkv + head, K|V): the
// slot's K rows [len][d] and its V blocks [ceil8(len)/8][d][8] are contiguous
// in the pool and are copied as they are, 16 bytes per lane.  Packed layout
// of slot i at byte base[i]: for l, h: K rows then V blocks.
__global__ void __launch_bounds__(256) kv_pack_kernel(int dir, const int32_t* __restrict__ slots,
        const int32_t* __restrict__ lens, const int64_t* __restrict__ base, KvPages kp, int Hkv,
        int rowbytes, int es, uint8_t* __restrict__ kslab, uint8_t* __restrict__ vslab, uint8_t* __restrict__ stage) {
    const int i = blockIdx.x, lh = blockIdx.y, kv = blockIdx.z;
    const int l = lh / Hkv, h = lh - l * Hkv;
    const int len = lens[i], len8 = (len + 7) / 8 * 8;
    const int rows = kv ? len8 : len;   // K rows, or V positions in whole 8-position blocks
    const size_t st_off = static_cast<size_t>(base[i]) +
                          (static_cast<size_t>(lh) * (len + len8) + (kv ? len : 0)) * rowbytes;
    u32x4* st = reinterpret_cast<u32x4*>(stage + st_off);
    const size_t per_row = static_cast<size_t>(rowbytes) / 16;
    // page by page (one page: every position of a contiguous slot); the rows
    // of a page are contiguous in both layouts (V: its 8-position blocks)
    for (int p0 = 0; p0 < rows; p0 += kp.page) {
        int lp;
        const int pid = kv_page(kp, slots[i], p0, &lp);
        const size_t pool_off = kv_block(kp, l, Hkv, pid, h) * es + static_cast<size_t>(lp) * rowbytes;
        u32x4* pool = reinterpret_cast<u32x4*>((kv ? vslab : kslab) + pool_off);
        const int n_rows = min(kp.page, rows - p0);
        const size_t n16 = static_cast<size_t>(n_rows) * per_row;
        u32x4* sp = st + static_cast<size_t>(p0) * per_row;
        for (size_t j = threadIdx.x; j < n16; j += blockDim.x) {
            if (dir == 0) sp[j] = pool[j];
            else pool[j] = sp[j];
        }
    }
}

hipError_t launch_kv_pack(int dir, const int32_t* slots, const int32_t* lens, const int64_t* base, int n, int L,
                          const KvPages& kp, int Hkv, int rowbytes, int es, void* kslab, void* vslab,
                          void* stage, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(kv_pack_kernel, dim3(n, L * Hkv, 2), dim3(256), 0, s, dir, slots, lens, base, kp, Hkv,
                       rowbytes, es, static_cast<uint8_t*>(kslab), static_cast<uint8_t*>(vslab),
                       static_cast<uint8_t*>(stage));
    return hipGetLastError();
}

// Plain streaming copy: 16 bytes per lane per iteration, grid-stride.
__global__ void __launch_bounds__(256) copy16_kernel(u32x4* __restrict__ dst,
        const u32x4* __restrict__ src, size_t n16) {
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
        dst[i] = src[i];
}

// Read-only stream: every thread XORs the 16-byte words it reads (four
// independent loads in flight per iteration) and each workgroup writes one
// word, so the kernel moves n16 * 16 bytes in and 4 bytes per workgroup out.
__global__ void __launch_bounds__(256) read16_kernel(const u32x4* __restrict__ src, size_t n16,
                                                     uint32_t* __restrict__ out) {
    __shared__ uint32_t red[4];
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    u32x4 acc = {0u, 0u, 0u, 0u};
    size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        acc ^= a ^ b ^ c ^ d;
    }
    for (; i < n16; i += stride) acc ^= src[i];
    uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
    for (int o = 32; o > 0; o >>= 1) x ^= static_cast<uint32_t>(__shfl_xor(static_cast<int>(x), o, 64));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) out[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

hipError_t launch_read16(const void* src, size_t n16, uint32_t* out, int n_blocks, hipStream_t s) {
    if (n_blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(read16_kernel, dim3(static_cast<unsigned>(n_blocks)), dim3(256), 0, s,
                       static_cast<const u32x4*>(src), n16, out);
    return hipGetLastError();
}

hipError_t launch_copy16(void* dst, const void* src, size_t n16, hipStream_t s) {
    if (n16 == 0) return hipSuccess;
    size_t blocks = (n16 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(copy16_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                       static_cast<u32x4*>(dst), static_cast<const u32x4*>(src), n16);
    return hipGetLastError();
}

}  // namespace rl
