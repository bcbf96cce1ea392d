// Kernels of the backward pass through the dense evaluation (binary32).
//
// The transformed network computes the same function as the strided network on
// every window (Theorem "processing chain", Sect. 4.3), so its gradients for a
// whole image are obtained by backpropagating through its own steps in reverse;
// the paper notes (Sect. 6.2, fine-tuning on entire images) that the gradients
// of Stuff and Trim are trivial, that Frag and Defrag are inverse permutations
// of each other, and that the sliding max-pool needs only elementary calculus.
//
//  frag_scatter_grad   transpose of Defrag_{k*_L} + Trim: the upstream gradient
//                      of the dense output [C][O_h][O_w] written into the final
//                      fragment layout [F][U_h][U_w][C] (zero for the trimmed
//                      positions).
//  pool_frag_backward  transpose of Frag_k after the sliding max-pool, fused with
//                      the activation's derivative: every pool input sample
//                      gathers the gradients of the (at most k_h k_w) sliding
//                      windows whose maximum it is.  The maximum of a window is
//                      its first maximal sample in row-major order, the rule the
//                      strided network's max-pool gradient uses too.
//  act_backward        dy = g * act'(a) for a convolution without a pool.
//  pad_grad            zero border of fh-1 x fw-1 around every fragment: the input
//                      gradient is then a valid convolution with the transposed,
//                      flipped filters (the forward convolution kernels run it).
//  wgrad_mfma          dW[o][i][t] = sum_p dy[p][o] x[p + t][i]: per tap a GEMM
//                      over all output positions p of all fragments (MFMA
//                      32x32x2 binary32, split over p, partial sums reduced in a
//                      fixed order by wgrad_reduce).
//  bias_partial/reduce db[o] = sum_p dy[p][o], two fixed-order passes.
//  crop_to_planar      transpose of Stuff: the stuffed input's gradient cropped
//                      to the signal and written planar.
#include <algorithm>
#include <mutex>
#include <vector>

#include "dev_common.h"
#include "dss_internal.h"

namespace dss {

constexpr int kBT = 256;

// ------------------------------------------------------------------ frag_scatter_grad
__global__ __launch_bounds__(kBT) void frag_scatter_grad_kernel(const float* __restrict__ g, int C, int O_h, int O_w,
                                                               int K_h, int K_w, int U_h, int U_w,
                                                               float* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kBT + threadIdx.x;
    const int64_t per = (int64_t)U_h * U_w;
    if (p >= (int64_t)K_h * K_w * per) return;
    const int f = (int)(p / per);
    const int q = (int)(p % per);
    const int y = q / U_w, x = q % U_w;
    const int i = y * K_h + f / K_w, j = x * K_w + f % K_w;    // dense position of this fragment sample
    const bool in = i < O_h && j < O_w;
    float* o = out + p * C;
    for (int c = 0; c < C; ++c) o[c] = in ? g[((int64_t)c * O_h + i) * O_w + j] : 0.f;
}

hipError_t launch_frag_scatter_grad(const float* g, int C, int O_h, int O_w, int K_h, int K_w, int U_h, int U_w,
                                    float* out, hipStream_t s) {
    const int64_t n = (int64_t)K_h * K_w * U_h * U_w;
    frag_scatter_grad_kernel<<<dim3((unsigned)ceil_div64(n, kBT)), kBT, 0, s>>>(g, C, O_h, O_w, K_h, K_w, U_h, U_w, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ activation derivative
__device__ __forceinline__ float act_grad(int act, float a) {
    if (act == DSS_ACT_RELU) return a > 0.f ? 1.f : 0.f;
    if (act == DSS_ACT_TANH) return 1.f - a * a;
    return 1.f;
}

// ------------------------------------------------------------------ pool_frag_backward
// One thread per (input fragment, pool-input sample, group of V channels).
template <int V>
__global__ __launch_bounds__(kBT) void pool_frag_backward_kernel(const float* __restrict__ g,
                                                                const float* __restrict__ a, int S_h, int S_w,
                                                                int E_h, int E_w, int C, int k_h, int k_w, int act,
                                                                float* __restrict__ out) {
    const int CV = C / V;
    const int P_h = E_h - k_h + 1, P_w = E_w - k_w + 1;      // sliding-pool extents
    const int U_h = P_h / k_h, U_w = P_w / k_w;
    const int64_t total = (int64_t)S_h * S_w * E_h * E_w * CV;
    const int64_t idx = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (idx >= total) return;
    const int cv = (int)(idx % CV);
    int64_t t = idx / CV;
    const int x = (int)(t % E_w);
    t /= E_w;
    const int y = (int)(t % E_h);
    const int s = (int)(t / E_h);
    const int b_h = s / S_w, b_w = s % S_w;
    const float* frag = a + (int64_t)s * E_h * E_w * C + cv * V;

    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;
    for (int dy = 0; dy < k_h; ++dy) {
        const int py = y - dy;
        if (py < 0 || py >= P_h) continue;
        for (int dx = 0; dx < k_w; ++dx) {
            const int px = x - dx;
            if (px < 0 || px >= P_w) continue;
            // first maximum of window (py, px), per channel
            float best[V];
            int arg[V];
            VecIO<float, V>::load(frag + ((int64_t)py * E_w + px) * C, best);
#pragma unroll
            for (int e = 0; e < V; ++e) arg[e] = 0;
            for (int a2 = 0; a2 < k_h; ++a2)
                for (int b2 = 0; b2 < k_w; ++b2) {
                    if ((a2 | b2) == 0) continue;
                    float v[V];
                    VecIO<float, V>::load(frag + ((int64_t)(py + a2) * E_w + px + b2) * C, v);
#pragma unroll
                    for (int e = 0; e < V; ++e)
                        if (v[e] > best[e]) {
                            best[e] = v[e];
                            arg[e] = a2 * k_w + b2;
                        }
                }
            const int f_new = ((py % k_h) * S_h + b_h) * (k_w * S_w) + (px % k_w) * S_w + b_w;
            float gv[V];
            VecIO<float, V>::load(g + (((int64_t)f_new * U_h + py / k_h) * U_w + px / k_w) * C + cv * V, gv);
            const int me = dy * k_w + dx;
#pragma unroll
            for (int e = 0; e < V; ++e)
                if (arg[e] == me) acc[e] += gv[e];
        }
    }
    if (act != DSS_ACT_NONE) {
        float av[V];
        VecIO<float, V>::load(frag + ((int64_t)y * E_w + x) * C, av);
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] *= act_grad(act, av[e]);
    }
    VecIO<float, V>::store(out + (((int64_t)s * E_h + y) * E_w + x) * C + cv * V, acc);
}

hipError_t launch_pool_frag_backward(const float* g, const float* a, int S_h, int S_w, int E_h, int E_w, int C,
                                     int k_h, int k_w, int act, float* out, hipStream_t s) {
    const int64_t n = (int64_t)S_h * S_w * E_h * E_w;
    if (C % 4 == 0) {
        pool_frag_backward_kernel<4><<<dim3((unsigned)ceil_div64(n * (C / 4), kBT)), kBT, 0, s>>>(
            g, a, S_h, S_w, E_h, E_w, C, k_h, k_w, act, out);
    } else {
        pool_frag_backward_kernel<1><<<dim3((unsigned)ceil_div64(n * C, kBT)), kBT, 0, s>>>(
            g, a, S_h, S_w, E_h, E_w, C, k_h, k_w, act, out);
    }
    return hipGetLastError();
}

// ------------------------------------------------------------------ act_backward
__global__ __launch_bounds__(kBT) void act_backward_kernel(const float* __restrict__ g, const float* __restrict__ a,
                                                          int64_t n, int act, float* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (p < n) out[p] = g[p] * act_grad(act, a[p]);
}

hipError_t launch_act_backward(const float* g, const float* a, int64_t n, int act, float* out, hipStream_t s) {
    act_backward_kernel<<<dim3((unsigned)ceil_div64(n, kBT)), kBT, 0, s>>>(g, a, n, act, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ pad_grad
__global__ __launch_bounds__(kBT) void pad_grad_kernel(const float* __restrict__ in, int F, int E_h, int E_w, int C,
                                                      int p_h, int p_w, float* __restrict__ out) {
    const int Wp = E_w + 2 * p_w, Hp = E_h + 2 * p_h;
    const int64_t total = (int64_t)F * Hp * Wp * C;
    const int64_t idx = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (idx >= total) return;
    const int c = (int)(idx % C);
    int64_t t = idx / C;
    const int x = (int)(t % Wp) - p_w;
    t /= Wp;
    const int y = (int)(t % Hp) - p_h;
    const int64_t f = t / Hp;
    const bool in_range = y >= 0 && y < E_h && x >= 0 && x < E_w;
    out[idx] = in_range ? in[((f * E_h + y) * E_w + x) * C + c] : 0.f;
}

hipError_t launch_pad_grad(const float* in, int F, int E_h, int E_w, int C, int p_h, int p_w, float* out,
                           hipStream_t s) {
    const int64_t n = (int64_t)F * (E_h + 2 * p_h) * (E_w + 2 * p_w) * C;
    pad_grad_kernel<<<dim3((unsigned)ceil_div64(n, kBT)), kBT, 0, s>>>(in, F, E_h, E_w, C, p_h, p_w, out);
    return hipGetLastError();
}

// ------------------------------------------------------------------ wgrad (MFMA)
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWM = 128;              // workgroup tile: output channels
constexpr int kKC = 32;               // positions per chunk
constexpr int kWP = 160;              // LDS row pitch in floats: 128 + 32, so the two half-waves
                                      // of a read hit disjoint banks
constexpr size_t kWgradLds = 2 * 2 * kKC * kWP * sizeof(float);

// Workgroup (o tile, i tile, tap, split): 4 waves in a 2 x 2 grid, each a
// 64 x (32 NTW) block of MFMA 32x32x2 tiles, so the workgroup covers 128 output
// channels and 64 NTW input channels (NTW = 1 for layers with at most 64 input
// channels).  The output positions p of all fragments are numbered row-major
// (fragment, row, column); chunk c holds positions 32c .. 32c + 31 and split s
// takes chunks [c0, c1).  Position p's gradient row is dy[p]; its input sample
// for tap (t_h, t_w) is x[f][y + t_h][x + t_w].
template <bool VEC, int NTW>
__global__ __launch_bounds__(256) void wgrad_mfma_kernel(const float* __restrict__ dy, const float* __restrict__ x,
                                                        int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                                                        int fh, int fw, int64_t P, int64_t nchunks, int otiles,
                                                        int itiles, int splits, float* __restrict__ partial) {
    constexpr int BNW = 64 * NTW;                 // input channels per workgroup
    constexpr int TPR = BNW / 4;                  // staging threads per B row (4 channels each)
    constexpr int RPP = 256 / TPR;                // B rows per staging pass
    constexpr int BPASS = kKC / RPP;
    extern __shared__ __attribute__((aligned(16))) float wl[];
    // A (output-gradient) chunks in buffers 0/1, B (input) chunks in buffers 2/3
    auto lds_buf = [&](int k) { return wl + k * (kKC * kWP); };
    // Workgroups are handed to the 8 XCDs round-robin by id; remap so that every
    // XCD runs one contiguous range of the logical order (o tile, i tile, tap
    // fastest, split slowest): the workgroups on an XCD then read the same chunks
    // of dy and x from its L2.
    const int total = gridDim.x;
    const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int q8 = total / 8, r8 = total % 8;
    int bid = xcd < r8 ? xcd * (q8 + 1) + slot : r8 * (q8 + 1) + (xcd - r8) * q8 + slot;
    const int ot = bid % otiles;
    bid /= otiles;
    const int it = bid % itiles;
    bid /= itiles;
    const int taps = fh * fw;
    const int tap = bid % taps;
    const int split = bid / taps;
    const int th = tap / fw, tw = tap % fw;
    const int64_t c0 = nchunks * split / splits, c1 = nchunks * (split + 1) / splits;
    const int o0 = ot * kWM, i0 = it * BNW;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1, half = lane >> 5, l32 = lane & 31;
    const int a_col = (tid & 31) * 4, a_row = tid >> 5;        // A staging: rows a_row + 8 k
    const int b_col = (tid % TPR) * 4, b_row = tid / TPR;      // B staging: rows b_row + RPP k
    const int64_t plane = (int64_t)E_h * E_w;

    floatx16 acc[2][NTW];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < NTW; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

    float4 ra[4], rb[BPASS];
    auto load4 = [&](const float* base, int c_lo, int C, bool ok) -> float4 {
        if (!ok) return make_float4(0.f, 0.f, 0.f, 0.f);
        if (VEC) return c_lo + 3 < C ? *reinterpret_cast<const float4*>(base + c_lo) : make_float4(0.f, 0.f, 0.f, 0.f);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = c_lo + e < C ? base[c_lo + e] : 0.f;
        return make_float4(v[0], v[1], v[2], v[3]);
    };
    auto load_chunk = [&](int64_t c) {
        const int64_t pc = c * kKC;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int64_t p = pc + a_row + 8 * k;
            ra[k] = load4(dy + p * Cout, o0 + a_col, Cout, p < P);
        }
#pragma unroll
        for (int k = 0; k < BPASS; ++k) {
            const int64_t p = pc + b_row + RPP * k;
            const int64_t f = p / plane;
            const int r = (int)(p - f * plane);
            const int y = r / E_w, xx = r - y * E_w;
            rb[k] = load4(x + ((f * U_h + y + th) * U_w + xx + tw) * Cin, i0 + b_col, Cin, p < P);
        }
    };
    auto store_chunk = [&](int buf) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            *reinterpret_cast<float4*>(lds_buf(buf) + (a_row + 8 * k) * kWP + a_col) = ra[k];
#pragma unroll
        for (int k = 0; k < BPASS; ++k)
            *reinterpret_cast<float4*>(lds_buf(2 + buf) + (b_row + RPP * k) * kWP + b_col) = rb[k];
    };

    if (c0 < c1) {
        load_chunk(c0);
        store_chunk(0);
    }
    __syncthreads();
    for (int64_t c = c0; c < c1; ++c) {
        const int buf = (int)((c - c0) & 1);
        const bool more = c + 1 < c1;
        if (more) load_chunk(c + 1);
        const float* A = lds_buf(buf);
        const float* Bm = lds_buf(2 + buf);
#pragma unroll 4
        for (int ks = 0; ks < kKC / 2; ++ks) {
            const int p = 2 * ks + half;
            float av[2], bv[NTW];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt) av[mt] = A[p * kWP + wm * 64 + mt * 32 + l32];
#pragma unroll
            for (int nt = 0; nt < NTW; ++nt) bv[nt] = Bm[p * kWP + wn * 32 * NTW + nt * 32 + l32];
#pragma unroll
            for (int mt = 0; mt < 2; ++mt)
#pragma unroll
                for (int nt = 0; nt < NTW; ++nt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
        }
        if (more) store_chunk(buf ^ 1);
        __syncthreads();
    }

    // D[i][j] of a 32x32 tile sits in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    float* dst = partial + ((size_t)split * taps + tap) * Cout * Cin;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
            const int ii = i0 + wn * 32 * NTW + nt * 32 + l32;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int o = o0 + wm * 64 + mt * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
                if (o < Cout && ii < Cin) dst[(size_t)o * Cin + ii] = acc[mt][nt][v];
            }
        }
}

// dW[o][i][th][tw] = sum over splits (in order) of partial[s][tap][o][i].
__global__ __launch_bounds__(kBT) void wgrad_reduce_kernel(const float* __restrict__ partial, int splits, int taps,
                                                          int Cout, int Cin, float* __restrict__ dw) {
    const int64_t n = (int64_t)Cout * Cin * taps;
    const int64_t p = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (p >= n) return;
    const int tap = (int)(p % taps);
    const int64_t oi = p / taps;                 // o * Cin + i
    const int64_t stride = (int64_t)taps * Cout * Cin;
    const float* src = partial + (int64_t)tap * Cout * Cin + oi;
    float s = 0.f;
    for (int k = 0; k < splits; ++k) s += src[k * stride];
    dw[p] = s;                                   // [o][i][th][tw] with tap = th * fw + tw
}

static hipError_t allow_lds(const void* kern, size_t lds) {
    if (lds <= 64 * 1024) return hipSuccess;
    static std::mutex mu;
    static std::vector<const void*> done;
    std::lock_guard<std::mutex> lock(mu);
    for (const void* k : done)
        if (k == kern) return hipSuccess;
    hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess) done.push_back(kern);
    return e;
}

WgradPlan wgrad_plan(int F, int E_h, int E_w, int Cout, int Cin, int fh, int fw) {
    WgradPlan w;
    w.ntw = Cin <= 64 ? 1 : 2;
    w.positions = (int64_t)F * E_h * E_w;
    w.nchunks = (w.positions + kKC - 1) / kKC;
    w.otiles = (Cout + kWM - 1) / kWM;
    w.itiles = (Cin + 64 * w.ntw - 1) / (64 * w.ntw);
    const int64_t base = (int64_t)w.otiles * w.itiles * fh * fw;
    // Two workgroups fit a CU (80 KB of LDS each), 512 run at once.  Take at
    // least eight rounds of 512 workgroups and, among the split counts up to
    // twice that, the one whose last round is fullest; every split keeps at least
    // 8 chunks.
    const int64_t max_splits = std::max<int64_t>(1, std::min<int64_t>(4096, w.nchunks / 8));
    const int64_t lo = std::min(max_splits, std::max<int64_t>(1, (512 * 8 + base - 1) / base));
    const int64_t hi = std::min(max_splits, 2 * lo);
    int64_t best = lo;
    double best_fill = -1.0;
    for (int64_t sp = lo; sp <= hi; ++sp) {
        const int64_t total = base * sp;
        const double fill = (double)total / (double)(((total + 511) / 512) * 512);
        if (fill > best_fill + 1e-9) {
            best_fill = fill;
            best = sp;
        }
    }
    w.splits = (int)best;
    w.partial_floats = (int64_t)w.splits * fh * fw * Cout * Cin;
    return w;
}

template <bool VEC, int NTW>
static hipError_t run_wgrad(const float* dy, const float* x, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                            int fh, int fw, const WgradPlan& w, float* partial, hipStream_t s) {
    auto kern = wgrad_mfma_kernel<VEC, NTW>;
    hipError_t e = allow_lds((const void*)kern, kWgradLds);
    if (e != hipSuccess) return e;
    const int64_t nblocks = (int64_t)w.otiles * w.itiles * fh * fw * w.splits;
    if (nblocks >= (1ll << 31)) return hipErrorInvalidConfiguration;
    kern<<<dim3((unsigned)nblocks), 256, kWgradLds, s>>>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w.positions,
                                                         w.nchunks, w.otiles, w.itiles, w.splits, partial);
    return hipGetLastError();
}

hipError_t launch_wgrad(const float* dy, const float* x, int F, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                        int fh, int fw, const WgradPlan& w, float* partial, float* dw, hipStream_t s) {
    (void)F;
    const bool vec = Cout % 4 == 0 && Cin % 4 == 0;
    hipError_t e;
    if (w.ntw == 1)
        e = vec ? run_wgrad<true, 1>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, s)
                : run_wgrad<false, 1>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, s);
    else
        e = vec ? run_wgrad<true, 2>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, s)
                : run_wgrad<false, 2>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, s);
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)Cout * Cin * fh * fw;
    wgrad_reduce_kernel<<<dim3((unsigned)ceil_div64(n, kBT)), kBT, 0, s>>>(partial, w.splits, fh * fw, Cout, Cin, dw);
    return hipGetLastError();
}

// ------------------------------------------------------------------ bias gradient
// Block b sums positions [b*P/nb, (b+1)*P/nb) for every channel (threads stride
// over channels); the reduce sums the blocks in order.
__global__ __launch_bounds__(kBT) void bias_partial_kernel(const float* __restrict__ dy, int64_t P, int C, int nb,
                                                          float* __restrict__ part) {
    const int b = blockIdx.x;
    const int64_t p0 = P * b / nb, p1 = P * (b + 1) / nb;
    for (int c = threadIdx.x; c < C; c += kBT) {
        float s = 0.f;
        for (int64_t p = p0; p < p1; ++p) s += dy[p * C + c];
        part[(int64_t)b * C + c] = s;
    }
}

__global__ __launch_bounds__(kBT) void bias_reduce_kernel(const float* __restrict__ part, int nb, int C,
                                                         float* __restrict__ db) {
    const int c = blockIdx.x * kBT + threadIdx.x;
    if (c >= C) return;
    float s = 0.f;
    for (int b = 0; b < nb; ++b) s += part[(int64_t)b * C + c];
    db[c] = s;
}

int bias_blocks(int64_t P) { return (int)std::max<int64_t>(1, std::min<int64_t>(2048, P / 256)); }

hipError_t launch_bias_grad(const float* dy, int64_t P, int C, float* part, float* db, hipStream_t s) {
    const int nb = bias_blocks(P);
    bias_partial_kernel<<<dim3((unsigned)nb), kBT, 0, s>>>(dy, P, C, nb, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    bias_reduce_kernel<<<dim3((unsigned)ceil_div64(C, kBT)), kBT, 0, s>>>(part, nb, C, db);
    return hipGetLastError();
}

// ------------------------------------------------------------------ crop_to_planar
__global__ __launch_bounds__(kBT) void crop_to_planar_kernel(const float* __restrict__ in, int D_w, int C, int H, int W,
                                                            float* __restrict__ out) {
    const int64_t p = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (p >= (int64_t)H * W) return;
    const int y = (int)(p / W), x = (int)(p % W);
    const float* src = in + ((int64_t)y * D_w + x) * C;
    for (int c = 0; c < C; ++c) out[(int64_t)c * H * W + p] = src[c];
}

hipError_t launch_crop_to_planar(const float* in, int D_w, int C, int H, int W, float* out, hipStream_t s) {
    crop_to_planar_kernel<<<dim3((unsigned)ceil_div64((int64_t)H * W, kBT)), kBT, 0, s>>>(in, D_w, C, H, W, out);
    return hipGetLastError();
}

}  // namespace dss
