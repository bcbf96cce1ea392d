// Data-movement kernels of the dense evaluation.  All are HBM-bound streaming
// kernels: no arithmetic besides the channel-wise maximum of the pool.
//
//  stuff_pack   Stuff_r per axis (Definition "stuff-trim", Sect. 4.3): copy the
//               planar [C][H][W] signal into the channels-last [D_h][D_w][C]
//               working layout and append r dummy samples (zeta = +0) at the end
//               of each axis.
//  pool_frag    Slide_{g_max} followed by Frag_k (Definition "processing chain",
//               Sect. 4.2): the k_h x k_w maximum at every position of every
//               fragment (stride 1), written straight to its fragment after
//               fragmentation.  Pools up to 4 rows high use the separable strip
//               kernel (each input row read once per column); taller pools the
//               direct one.  Per axis, sliding-pool sample m*k + a of input
//               fragment b lands at sample m of output fragment a*S + b
//               (Lemma "frag-ops", Sect. 4.1).
//  pool_stride  Stride_{g_max} of a relaxed layer (Definition "evalrelax",
//               appendix): the maximum over non-overlapping k_h x k_w blocks of
//               one channels-last signal, no fragmentation.  Every input sample
//               is read exactly once.
//  pool_dilate  Dilate_{(g_max, k*_{j-1})} of the dilated fashion (appendix,
//               Definition "dilate"): the maximum over k_h x k_w samples that are
//               dil samples apart, on one channels-last signal.
//  defrag_trim  Defrag_{k*_L} and Trim_r (appendix lemma on the simplified
//               defragmentation; Definition "stuff-trim"): dense output sample
//               (i, j) is sample (i div K_h, j div K_w) of fragment
//               (i mod K_h) * K_w + (j mod K_w); only i < H - B_h + 1,
//               j < W - B_w + 1 are written.  Output is planar binary32.
//  to_planar    channels-last fragments -> planar binary32 [F][C][h][w].
//  patch_pack   Subsignal extraction (Sect. 2.3) for the strided baseline: the
//               B_h x B_w windows with row-major indices first..first+count-1
//               copied to a channels-last fragment batch [count][B_h][B_w][C].
//  window_scatter  the strided baseline's per-window outputs [count][C] written
//               to their places in the planar binary32 dense output grid.
//  frag_planar  dss_frag / dss_defrag on planar tensors (pure permutations of
//               2- or 4-byte elements).
#include "dev_common.h"
#include "dss_internal.h"

namespace dss {

constexpr int kThreads = 256;

// ------------------------------------------------------------------ stuff_pack
template <typename E>
__global__ __launch_bounds__(kThreads) void stuff_pack_kernel(const E* __restrict__ in, int C, int H, int W,
                                                             E* __restrict__ out, int D_h, int D_w) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= (int64_t)D_h * D_w) return;
    const int y = (int)(p / D_w), x = (int)(p % D_w);
    E* o = out + p * C;
    if (y < H && x < W) {
        for (int c = 0; c < C; ++c) o[c] = in[((int64_t)c * H + y) * W + x];
    } else {
        for (int c = 0; c < C; ++c) o[c] = E(0);
    }
}

hipError_t launch_stuff_pack(dss_dtype dt, const void* in, int C, int H, int W, void* out, int D_h, int D_w,
                             hipStream_t s) {
    const int64_t n = (int64_t)D_h * D_w;
    const dim3 grid((unsigned)ceil_div64(n, kThreads));
    if (dt == DSS_BF16)
        stuff_pack_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, C, H, W, (uint16_t*)out, D_h, D_w);
    else
        stuff_pack_kernel<uint32_t><<<grid, kThreads, 0, s>>>((const uint32_t*)in, C, H, W, (uint32_t*)out, D_h, D_w);
    return hipGetLastError();
}

// ------------------------------------------------------------------ pool_frag
// One thread per (input fragment, sliding-pool position, group of V channels).
template <typename T, int V>
__global__ __launch_bounds__(kThreads) void pool_frag_kernel(const T* __restrict__ in, int S_h, int S_w, int E_h,
                                                            int E_w, int C, int k_h, int k_w, T* __restrict__ out,
                                                            int U_h, int U_w) {
    const int CV = C / V;
    const int P_h = k_h * U_h, P_w = k_w * U_w;   // sliding-pool extents
    const int64_t total = (int64_t)S_h * S_w * P_h * P_w * CV;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    int64_t t = idx / CV;
    const int x = (int)(t % P_w);
    t /= P_w;
    const int y = (int)(t % P_h);
    const int s = (int)(t / P_h);
    const int b_h = s / S_w, b_w = s % S_w;

    const T* src = in + (((int64_t)s * E_h + y) * E_w + x) * C + cv * V;
    float m[V];
    VecIO<T, V>::load(src, m);
    for (int dy = 0; dy < k_h; ++dy) {
        for (int dx = 0; dx < k_w; ++dx) {
            if ((dy | dx) == 0) continue;
            float v[V];
            VecIO<T, V>::load(src + ((int64_t)dy * E_w + dx) * C, v);
#pragma unroll
            for (int e = 0; e < V; ++e) m[e] = fmaxf(m[e], v[e]);
        }
    }
    const int a_h = y % k_h, a_w = x % k_w;
    const int f_new = (a_h * S_h + b_h) * (k_w * S_w) + (a_w * S_w + b_w);
    T* dst = out + (((int64_t)f_new * U_h + y / k_h) * U_w + x / k_w) * C + cv * V;
    VecIO<T, V>::store(dst, m);
}

// Separable form for small pool heights: one thread per (input fragment, strip
// of NY sliding-pool rows, column, group of V channels).  The thread walks the
// KH + NY - 1 input rows of its strip once, keeps the horizontal maxima of the
// last KH rows in registers, and emits one output row per input row.
template <typename T, int V, int KH, int NY>
__global__ __launch_bounds__(kThreads) void pool_frag_strip_kernel(const T* __restrict__ in, int S_h, int S_w,
                                                                  int E_h, int E_w, int C, int k_w,
                                                                  T* __restrict__ out, int U_h, int U_w) {
    const int CV = C / V;
    const int P_h = KH * U_h, P_w = k_w * U_w;
    const int strips = (P_h + NY - 1) / NY;
    const int64_t total = (int64_t)S_h * S_w * strips * P_w * CV;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    int64_t t = idx / CV;
    const int x = (int)(t % P_w);
    t /= P_w;
    const int strip = (int)(t % strips);
    const int s = (int)(t / strips);
    const int b_h = s / S_w, b_w = s % S_w;
    const int y0 = strip * NY;
    const int y1 = min(y0 + NY, P_h);

    const T* src = in + (((int64_t)s * E_h + y0) * E_w + x) * C + cv * V;
    const int a_w = x % k_w;
    const int Fw = k_w * S_w;
    const int64_t row_stride = (int64_t)E_w * C;
    float ring[KH][V];
    for (int yy = y0; yy < y1 + KH - 1; ++yy, src += row_stride) {
        float h[V];
        VecIO<T, V>::load(src, h);
        for (int dx = 1; dx < k_w; ++dx) {
            float v[V];
            VecIO<T, V>::load(src + (int64_t)dx * C, v);
#pragma unroll
            for (int e = 0; e < V; ++e) h[e] = fmaxf(h[e], v[e]);
        }
#pragma unroll
        for (int r = 0; r + 1 < KH; ++r)
#pragma unroll
            for (int e = 0; e < V; ++e) ring[r][e] = ring[r + 1][e];
#pragma unroll
        for (int e = 0; e < V; ++e) ring[KH - 1][e] = h[e];
        if (yy >= y0 + KH - 1) {
            const int y = yy - (KH - 1);
            float m[V];
#pragma unroll
            for (int e = 0; e < V; ++e) {
                m[e] = ring[0][e];
#pragma unroll
                for (int r = 1; r < KH; ++r) m[e] = fmaxf(m[e], ring[r][e]);
            }
            const int f_new = ((y % KH) * S_h + b_h) * Fw + (a_w * S_w + b_w);
            VecIO<T, V>::store(out + (((int64_t)f_new * U_h + y / KH) * U_w + x / k_w) * C + cv * V, m);
        }
    }
}

template <typename T, int V>
static void run_pool(const void* in, int S_h, int S_w, int E_h, int E_w, int C, int k_h, int k_w, void* out,
                     hipStream_t s) {
    const int U_h = (E_h - k_h + 1) / k_h, U_w = (E_w - k_w + 1) / k_w;
    constexpr int NY = 16;
    if (k_h >= 1 && k_h <= 4) {
        const int64_t total = (int64_t)S_h * S_w * ((k_h * U_h + NY - 1) / NY) * (k_w * U_w) * (C / V);
        const dim3 grid((unsigned)ceil_div64(total, kThreads));
        switch (k_h) {
            case 1: pool_frag_strip_kernel<T, V, 1, NY><<<grid, kThreads, 0, s>>>((const T*)in, S_h, S_w, E_h, E_w, C, k_w, (T*)out, U_h, U_w); break;
            case 2: pool_frag_strip_kernel<T, V, 2, NY><<<grid, kThreads, 0, s>>>((const T*)in, S_h, S_w, E_h, E_w, C, k_w, (T*)out, U_h, U_w); break;
            case 3: pool_frag_strip_kernel<T, V, 3, NY><<<grid, kThreads, 0, s>>>((const T*)in, S_h, S_w, E_h, E_w, C, k_w, (T*)out, U_h, U_w); break;
            default: pool_frag_strip_kernel<T, V, 4, NY><<<grid, kThreads, 0, s>>>((const T*)in, S_h, S_w, E_h, E_w, C, k_w, (T*)out, U_h, U_w); break;
        }
        return;
    }
    const int64_t total = (int64_t)S_h * S_w * (k_h * U_h) * (k_w * U_w) * (C / V);
    pool_frag_kernel<T, V><<<dim3((unsigned)ceil_div64(total, kThreads)), kThreads, 0, s>>>(
        (const T*)in, S_h, S_w, E_h, E_w, C, k_h, k_w, (T*)out, U_h, U_w);
}

hipError_t launch_pool_frag(dss_dtype dt, const void* in, int S_h, int S_w, int E_h, int E_w, int C, int k_h,
                            int k_w, void* out, hipStream_t s) {
    if (dt == DSS_BF16) {
        if (C % 8 == 0) run_pool<uint16_t, 8>(in, S_h, S_w, E_h, E_w, C, k_h, k_w, out, s);
        else if (C % 4 == 0) run_pool<uint16_t, 4>(in, S_h, S_w, E_h, E_w, C, k_h, k_w, out, s);
        else run_pool<uint16_t, 1>(in, S_h, S_w, E_h, E_w, C, k_h, k_w, out, s);
    } else {
        if (C % 4 == 0) run_pool<float, 4>(in, S_h, S_w, E_h, E_w, C, k_h, k_w, out, s);
        else run_pool<float, 1>(in, S_h, S_w, E_h, E_w, C, k_h, k_w, out, s);
    }
    return hipGetLastError();
}

// ------------------------------------------------------------------ pool_stride
// One thread per (output position, group of V channels); consecutive threads
// take consecutive channel groups, then consecutive output columns.
template <typename T, int V>
__global__ __launch_bounds__(kThreads) void pool_stride_kernel(const T* __restrict__ in, int E_w, int C, int k_h,
                                                              int k_w, T* __restrict__ out, int U_h, int U_w) {
    const int CV = C / V;
    const int64_t total = (int64_t)U_h * U_w * CV;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    const int64_t t = idx / CV;
    const int x = (int)(t % U_w);
    const int y = (int)(t / U_w);
    const T* src = in + ((int64_t)y * k_h * E_w + (int64_t)x * k_w) * C + cv * V;
    float m[V];
    VecIO<T, V>::load(src, m);
    for (int dy = 0; dy < k_h; ++dy) {
        for (int dx = 0; dx < k_w; ++dx) {
            if ((dy | dx) == 0) continue;
            float v[V];
            VecIO<T, V>::load(src + ((int64_t)dy * E_w + dx) * C, v);
#pragma unroll
            for (int e = 0; e < V; ++e) m[e] = fmaxf(m[e], v[e]);
        }
    }
    VecIO<T, V>::store(out + t * C + cv * V, m);
}

template <typename T, int V>
static void run_pool_stride(const void* in, int E_h, int E_w, int C, int k_h, int k_w, void* out, hipStream_t s) {
    const int U_h = E_h / k_h, U_w = E_w / k_w;
    const int64_t total = (int64_t)U_h * U_w * (C / V);
    if (total == 0) return;
    pool_stride_kernel<T, V><<<dim3((unsigned)ceil_div64(total, kThreads)), kThreads, 0, s>>>(
        (const T*)in, E_w, C, k_h, k_w, (T*)out, U_h, U_w);
}

hipError_t launch_pool_stride(dss_dtype dt, const void* in, int E_h, int E_w, int C, int k_h, int k_w, void* out,
                              hipStream_t s) {
    if (dt == DSS_BF16) {
        if (C % 8 == 0) run_pool_stride<uint16_t, 8>(in, E_h, E_w, C, k_h, k_w, out, s);
        else if (C % 4 == 0) run_pool_stride<uint16_t, 4>(in, E_h, E_w, C, k_h, k_w, out, s);
        else run_pool_stride<uint16_t, 1>(in, E_h, E_w, C, k_h, k_w, out, s);
    } else {
        if (C % 4 == 0) run_pool_stride<float, 4>(in, E_h, E_w, C, k_h, k_w, out, s);
        else run_pool_stride<float, 1>(in, E_h, E_w, C, k_h, k_w, out, s);
    }
    return hipGetLastError();
}

// ------------------------------------------------------------------ pool_dilate
template <typename T, int V>
__global__ __launch_bounds__(kThreads) void pool_dilate_kernel(const T* __restrict__ in, int E_w, int C, int k_h,
                                                              int k_w, int dil_h, int dil_w, T* __restrict__ out,
                                                              int P_h, int P_w) {
    const int CV = C / V;
    const int64_t total = (int64_t)P_h * P_w * CV;
    const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    const int64_t t = idx / CV;
    const int x = (int)(t % P_w);
    const int y = (int)(t / P_w);
    const T* src = in + ((int64_t)y * E_w + x) * C + cv * V;
    float m[V];
    VecIO<T, V>::load(src, m);
    for (int a = 0; a < k_h; ++a) {
        for (int b = 0; b < k_w; ++b) {
            if ((a | b) == 0) continue;
            float v[V];
            VecIO<T, V>::load(src + ((int64_t)a * dil_h * E_w + (int64_t)b * dil_w) * C, v);
#pragma unroll
            for (int e = 0; e < V; ++e) m[e] = fmaxf(m[e], v[e]);
        }
    }
    VecIO<T, V>::store(out + t * C + cv * V, m);
}

template <typename T, int V>
static void run_pool_dilate(const void* in, int E_h, int E_w, int C, int k_h, int k_w, int dh, int dw, void* out,
                            hipStream_t s) {
    const int P_h = E_h - dh * (k_h - 1), P_w = E_w - dw * (k_w - 1);
    const int64_t total = (int64_t)P_h * P_w * (C / V);
    if (total <= 0) return;
    pool_dilate_kernel<T, V><<<dim3((unsigned)ceil_div64(total, kThreads)), kThreads, 0, s>>>(
        (const T*)in, E_w, C, k_h, k_w, dh, dw, (T*)out, P_h, P_w);
}

hipError_t launch_pool_dilate(dss_dtype dt, const void* in, int E_h, int E_w, int C, int k_h, int k_w, int dil_h,
                              int dil_w, void* out, hipStream_t s) {
    if (dt == DSS_BF16) {
        if (C % 8 == 0) run_pool_dilate<uint16_t, 8>(in, E_h, E_w, C, k_h, k_w, dil_h, dil_w, out, s);
        else if (C % 4 == 0) run_pool_dilate<uint16_t, 4>(in, E_h, E_w, C, k_h, k_w, dil_h, dil_w, out, s);
        else run_pool_dilate<uint16_t, 1>(in, E_h, E_w, C, k_h, k_w, dil_h, dil_w, out, s);
    } else {
        if (C % 4 == 0) run_pool_dilate<float, 4>(in, E_h, E_w, C, k_h, k_w, dil_h, dil_w, out, s);
        else run_pool_dilate<float, 1>(in, E_h, E_w, C, k_h, k_w, dil_h, dil_w, out, s);
    }
    return hipGetLastError();
}

// ------------------------------------------------------------------ defrag_trim
template <typename T>
__global__ __launch_bounds__(kThreads) void defrag_trim_kernel(const T* __restrict__ in, int K_h, int K_w, int U_h,
                                                              int U_w, int C, float* __restrict__ out, int O_h,
                                                              int O_w) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= (int64_t)O_h * O_w) return;
    const int i = (int)(p / O_w), j = (int)(p % O_w);
    const int f = (i % K_h) * K_w + (j % K_w);
    const T* src = in + (((int64_t)f * U_h + i / K_h) * U_w + j / K_w) * C;
    for (int c = 0; c < C; ++c) out[(int64_t)c * O_h * O_w + p] = to_f32(src[c]);
}

hipError_t launch_defrag_trim(dss_dtype dt, const void* in, int K_h, int K_w, int U_h, int U_w, int C, float* out,
                              int O_h, int O_w, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div64((int64_t)O_h * O_w, kThreads));
    if (dt == DSS_BF16)
        defrag_trim_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, K_h, K_w, U_h, U_w, C, out, O_h, O_w);
    else
        defrag_trim_kernel<float><<<grid, kThreads, 0, s>>>((const float*)in, K_h, K_w, U_h, U_w, C, out, O_h, O_w);
    return hipGetLastError();
}

// The final step after a folded 1x1 convolution: the partial projections of
// the channel groups ([nbs][sample][4] binary32, `stride` floats apart) summed in
// group order, then the projection's bias and activation, for channels c < C.
__device__ __forceinline__ void sum_projection(const float* __restrict__ src, int64_t stride, int nbs, int C,
                                               const float* __restrict__ bias, int act, float* __restrict__ out,
                                               int64_t plane) {
    float4 a = *reinterpret_cast<const float4*>(src);
    for (int nb = 1; nb < nbs; ++nb) {
        const float4 b = *reinterpret_cast<const float4*>(src + nb * stride);
        a.x += b.x;
        a.y += b.y;
        a.z += b.z;
        a.w += b.w;
    }
    const float v[4] = {a.x, a.y, a.z, a.w};
    for (int c = 0; c < C; ++c) out[c * plane] = activate(act, v[c] + bias[c]);
}

// Defrag + Trim of the partial projections (the defrag_trim map).
__global__ __launch_bounds__(kThreads) void defrag_sum_kernel(const float* __restrict__ part, int64_t stride, int nbs,
                                                             int K_h, int K_w, int U_h, int U_w, int C,
                                                             const float* __restrict__ bias, int act,
                                                             float* __restrict__ out, int O_h, int O_w) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= (int64_t)O_h * O_w) return;
    const int i = (int)(p / O_w), j = (int)(p % O_w);
    const int f = (i % K_h) * K_w + (j % K_w);
    sum_projection(part + (((int64_t)f * U_h + i / K_h) * U_w + j / K_w) * 4, stride, nbs, C, bias, act, out + p,
                   (int64_t)O_h * O_w);
}

// The strided baseline's per-window outputs (the window_scatter map) from partial projections.
__global__ __launch_bounds__(kThreads) void window_scatter_sum_kernel(const float* __restrict__ part, int64_t stride,
                                                                     int nbs, int count, int C,
                                                                     const float* __restrict__ bias, int act,
                                                                     int64_t first, int64_t plane,
                                                                     float* __restrict__ out) {
    const int64_t n = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (n >= count) return;
    sum_projection(part + n * 4, stride, nbs, C, bias, act, out + first + n, plane);
}

// One signal of h x w samples (the dilated fashion's last layer) to planar, from partial projections.
__global__ __launch_bounds__(kThreads) void planar_sum_kernel(const float* __restrict__ part, int64_t stride, int nbs,
                                                             int64_t hw, int C, const float* __restrict__ bias,
                                                             int act, float* __restrict__ out) {
    const int64_t q = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (q >= hw) return;
    sum_projection(part + q * 4, stride, nbs, C, bias, act, out + q, hw);
}

hipError_t launch_defrag_sum(const float* part, int nbs, int K_h, int K_w, int U_h, int U_w, int C, const float* bias,
                             int act, float* out, int O_h, int O_w, hipStream_t s) {
    if (C < 1 || C > 4 || nbs < 1) return hipErrorInvalidValue;
    const dim3 grid((unsigned)ceil_div64((int64_t)O_h * O_w, kThreads));
    const int64_t stride = (int64_t)K_h * K_w * U_h * U_w * 4;
    defrag_sum_kernel<<<grid, kThreads, 0, s>>>(part, stride, nbs, K_h, K_w, U_h, U_w, C, bias, act, out, O_h, O_w);
    return hipGetLastError();
}

hipError_t launch_window_scatter_sum(const float* part, int nbs, int count, int C, const float* bias, int act,
                                     int64_t first, int64_t plane, float* out, hipStream_t s) {
    if (C < 1 || C > 4 || nbs < 1) return hipErrorInvalidValue;
    const dim3 grid((unsigned)ceil_div64(count, kThreads));
    window_scatter_sum_kernel<<<grid, kThreads, 0, s>>>(part, (int64_t)count * 4, nbs, count, C, bias, act, first,
                                                        plane, out);
    return hipGetLastError();
}

hipError_t launch_planar_sum(const float* part, int nbs, int h, int w, int C, const float* bias, int act, float* out,
                             hipStream_t s) {
    if (C < 1 || C > 4 || nbs < 1) return hipErrorInvalidValue;
    const int64_t hw = (int64_t)h * w;
    const dim3 grid((unsigned)ceil_div64(hw, kThreads));
    planar_sum_kernel<<<grid, kThreads, 0, s>>>(part, hw * 4, nbs, hw, C, bias, act, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ to_planar
template <typename T>
__global__ __launch_bounds__(kThreads) void to_planar_kernel(const T* __restrict__ in, int F, int h, int w, int C,
                                                            float* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t hw = (int64_t)h * w;
    if (p >= (int64_t)F * hw) return;
    const int64_t f = p / hw, q = p % hw;
    const T* src = in + p * C;
    for (int c = 0; c < C; ++c) out[(f * C + c) * hw + q] = to_f32(src[c]);
}

hipError_t launch_to_planar(dss_dtype dt, const void* in, int F, int h, int w, int C, float* out, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div64((int64_t)F * h * w, kThreads));
    if (dt == DSS_BF16)
        to_planar_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, F, h, w, C, out);
    else
        to_planar_kernel<float><<<grid, kThreads, 0, s>>>((const float*)in, F, h, w, C, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ patch_pack / window_scatter
template <typename E>
__global__ __launch_bounds__(kThreads) void patch_pack_kernel(const E* __restrict__ in, int C, int H, int W, int O_w,
                                                             int64_t first, int count, int B_h, int B_w,
                                                             E* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int64_t per = (int64_t)B_h * B_w;
    if (p >= (int64_t)count * per) return;
    const int64_t n = p / per;
    const int q = (int)(p % per);
    const int y = q / B_w, x = q % B_w;
    const int64_t win = first + n;
    const int i0 = (int)(win / O_w), j0 = (int)(win % O_w);
    const E* src = in + (int64_t)(i0 + y) * W + (j0 + x);
    E* o = out + p * C;
    for (int c = 0; c < C; ++c) o[c] = src[(int64_t)c * H * W];
}

hipError_t launch_patch_pack(dss_dtype dt, const void* in, int C, int H, int W, int O_w, int64_t first, int count,
                             int B_h, int B_w, void* out, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div64((int64_t)count * B_h * B_w, kThreads));
    if (dt == DSS_BF16)
        patch_pack_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, C, H, W, O_w, first, count, B_h,
                                                              B_w, (uint16_t*)out);
    else
        patch_pack_kernel<uint32_t><<<grid, kThreads, 0, s>>>((const uint32_t*)in, C, H, W, O_w, first, count, B_h,
                                                              B_w, (uint32_t*)out);
    return hipGetLastError();
}

// One thread per (channel, window): consecutive threads write consecutive
// output samples of one channel plane.
template <typename T>
__global__ __launch_bounds__(kThreads) void window_scatter_kernel(const T* __restrict__ in, int count, int C,
                                                                 int64_t first, int64_t plane,
                                                                 float* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= (int64_t)count * C) return;
    const int c = (int)(p / count);
    const int64_t n = p % count;
    out[(int64_t)c * plane + first + n] = to_f32(in[n * C + c]);
}

hipError_t launch_window_scatter(dss_dtype dt, const void* in, int count, int C, int64_t first, int64_t plane,
                                 float* out, hipStream_t s) {
    const dim3 grid((unsigned)ceil_div64((int64_t)count * C, kThreads));
    if (dt == DSS_BF16)
        window_scatter_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, count, C, first, plane, out);
    else
        window_scatter_kernel<float><<<grid, kThreads, 0, s>>>((const float*)in, count, C, first, plane, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ frag / defrag (planar)
// One thread per output element; consecutive threads write consecutive
// samples of one output row.
template <typename E>
__global__ __launch_bounds__(kThreads) void frag_planar_kernel(const E* __restrict__ in, int k_h, int k_w, int S_h,
                                                              int S_w, int C, int H, int W, E* __restrict__ out) {
    const int Ho = H / k_h, Wo = W / k_w;
    const int64_t total = (int64_t)k_h * S_h * k_w * S_w * C * Ho * Wo;
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= total) return;
    const int n = (int)(p % Wo);
    int64_t t = p / Wo;
    const int m = (int)(t % Ho);
    t /= Ho;
    const int c = (int)(t % C);
    const int fo = (int)(t / C);
    const int Fw = k_w * S_w;
    const int fh = fo / Fw, fw = fo % Fw;
    const int a_h = fh / S_h, b_h = fh % S_h, a_w = fw / S_w, b_w = fw % S_w;
    out[p] = in[(((int64_t)(b_h * S_w + b_w) * C + c) * H + (int64_t)m * k_h + a_h) * W + (int64_t)n * k_w + a_w];
}

template <typename E>
__global__ __launch_bounds__(kThreads) void defrag_planar_kernel(const E* __restrict__ in, int k_h, int k_w, int S_h,
                                                                int S_w, int C, int H, int W, E* __restrict__ out) {
    const int Y = H * k_h, X = W * k_w;
    const int64_t total = (int64_t)S_h * S_w * C * Y * X;
    const int64_t p = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (p >= total) return;
    const int x = (int)(p % X);
    int64_t t = p / X;
    const int y = (int)(t % Y);
    t /= Y;
    const int c = (int)(t % C);
    const int s = (int)(t / C);
    const int b_h = s / S_w, b_w = s % S_w;
    const int fo = ((y % k_h) * S_h + b_h) * (k_w * S_w) + (x % k_w) * S_w + b_w;
    out[p] = in[(((int64_t)fo * C + c) * H + y / k_h) * W + x / k_w];
}

hipError_t launch_frag_planar(int elem_bytes, bool inverse, const void* in, int k_h, int k_w, int S_h, int S_w, int C,
                              int H, int W, void* out, hipStream_t s) {
    const int64_t total = inverse ? (int64_t)S_h * S_w * C * H * k_h * W * k_w
                                  : (int64_t)k_h * S_h * k_w * S_w * C * (H / k_h) * (W / k_w);
    if (total == 0) return hipSuccess;
    const dim3 grid((unsigned)ceil_div64(total, kThreads));
    if (elem_bytes == 2) {
        if (inverse)
            defrag_planar_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, k_h, k_w, S_h, S_w, C, H, W, (uint16_t*)out);
        else
            frag_planar_kernel<uint16_t><<<grid, kThreads, 0, s>>>((const uint16_t*)in, k_h, k_w, S_h, S_w, C, H, W, (uint16_t*)out);
    } else {
        if (inverse)
            defrag_planar_kernel<uint32_t><<<grid, kThreads, 0, s>>>((const uint32_t*)in, k_h, k_w, S_h, S_w, C, H, W, (uint32_t*)out);
        else
            frag_planar_kernel<uint32_t><<<grid, kThreads, 0, s>>>((const uint32_t*)in, k_h, k_w, S_h, S_w, C, H, W, (uint32_t*)out);
    }
    return hipGetLastError();
}

}  // namespace dss
