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
//                      gradient is a valid convolution of the bordered gradient
//                      with the transposed, flipped filters.  The MFMA convolution
//                      reads the border virtually; this copy feeds the direct
//                      kernel (input gradients into few channels).
//  wgrad_mfma          dW[o][i][t] = sum_p dy[p][o] x[p + t][i]: per tap a GEMM
//                      over all output positions p of all fragments (MFMA
//                      32x32x2 binary32); a workgroup takes the taps of one
//                      filter row, which share their operand rows shifted by
//                      the tap; split over p, partial sums reduced in a fixed
//                      order by wgrad_reduce.  The same launch sums dy over p for
//                      the bias gradient db[o].
//  crop_to_planar      transpose of Stuff: the stuffed input's gradient cropped
//                      to the signal and written planar.
#include <algorithm>

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

constexpr int kWT = 64;               // workgroup tile: 64 output x 64 input channels
constexpr int kKC = 32;               // positions per chunk
constexpr int kWP = kWT + 32;         // LDS row pitch in floats: the two half-waves of a read
                                      // (rows p and p + 1) hit disjoint banks
constexpr int kMaxTT = 8;             // taps of one filter row per workgroup
constexpr int kMaxPackedTT = 4;       // MFMA tiles per wave in the packed (narrow-layer) mode

static size_t wgrad_lds_bytes(int tt) { return 2 * (size_t)(kKC + kKC + tt - 1) * kWP * sizeof(float); }

// Workgroup (o tile, i tile, tap row t_h, tap group, split) computes
//   dW[o][i][t_h][t_w] = sum_p dy[p][o] x[f][y + t_h][x + t_w][i]
// for 64 output channels, 64 input channels and the taps t_w of one group of up
// to TT consecutive taps of filter row t_h.  4 waves in a 2 x 2 grid, each a
// 32 x 32 MFMA tile per tap.
//
// Positions are numbered over the input width: q = (f E_h + y) U_w + x for
// x < U_w, of which x < E_w are output positions (dy row (f E_h + y) E_w + x)
// and the rest carry a zero gradient.  Then the input sample of tap (t_h, t_w)
// at q is the tap (t_h, 0) sample at q + t_w: within a row x + t_w < U_w for
// every output position.  A chunk of 32 positions therefore stages the dy rows
// of its 32 positions and the x rows of 32 + TT - 1 positions once, and every tap
// of the group reads its operand rows t_w further on in LDS -- TT times fewer
// global reads than one workgroup per tap.
//
// PACKED (layers with at most 32 input channels): the 64 columns of an MFMA
// tile hold g = 64 / cpt taps of cpt channels each (cpt: Cin rounded up to a
// power of two, at least 4), column j being tap j / cpt and channel j % cpt, so
// a narrow layer does not spend 64-column tiles on a few channels.  Tile t of a
// workgroup covers taps t g .. t g + g - 1 of its group; the staged x rows are
// cpt floats apart and column j of tap row q reads row q + j / cpt.
template <bool VEC, int TT, bool PACKED>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void wgrad_mfma_kernel(
    const float* __restrict__ dy, const float* __restrict__ x, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
    int fh, int fw, int Q, int nchunks, int otiles, int itiles, int ntg, int splits, int cpt,
    float* __restrict__ partial, float* __restrict__ bias_partial) {
    constexpr int RB = kKC + TT - 1;              // staged x rows per chunk (unpacked; bounds the buffer)
    extern __shared__ __attribute__((aligned(16))) float wl[];
    auto lds_a = [&](int buf) { return wl + buf * (kKC * kWP); };                  // dy rows
    auto lds_b = [&](int buf) { return wl + 2 * kKC * kWP + buf * (RB * kWP); };   // x rows
    // Workgroups are handed to the 8 XCDs round-robin by id; remap so that every
    // XCD runs one contiguous range of the logical order (o tile, i tile, tap
    // group, tap row fastest, split slowest): the workgroups on an XCD then read
    // the same chunks of dy and x from its L2.
    const int total = gridDim.x;
    const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int q8 = total / 8, r8 = total % 8;
    int bid = xcd < r8 ? xcd * (q8 + 1) + slot : r8 * (q8 + 1) + (xcd - r8) * q8 + slot;
    const int ot = bid % otiles;
    bid /= otiles;
    const int it = bid % itiles;
    bid /= itiles;
    const int tg = bid % ntg;
    bid /= ntg;
    const int th = bid % fh;
    const int split = bid / fh;
    const int g = PACKED ? kWT / cpt : 1;         // taps per MFMA tile
    const int span = TT * g;                      // taps per group
    const int tw0 = tg * span;
    const int ntt = min(span, fw - tw0);          // taps of this group
    const int rows_b = kKC + span - 1;            // staged x rows per chunk
    const int c0 = (int)((int64_t)nchunks * split / splits), c1 = (int)((int64_t)nchunks * (split + 1) / splits);
    const int o0 = ot * kWT, i0 = it * kWT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave & 1, wn = wave >> 1, half = lane >> 5, l32 = lane & 31;
    const int s_col = (tid & 15) * 4, s_row = tid >> 4;          // staging: 16 float4 per row, 16 rows per pass
    const int rowlen = E_h * U_w;                                // positions per fragment

    floatx16 acc[TT];
#pragma unroll
    for (int t = 0; t < TT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;

    float bsum = 0.f;   // sum of this lane's dy column over its positions (bias gradient)
    float4 ra[2], rb[3];
    auto load4 = [&](const float* base, int c_lo, int C, bool ok) -> float4 {
        if (!ok) return make_float4(0.f, 0.f, 0.f, 0.f);
        if (VEC) return c_lo + 3 < C ? *reinterpret_cast<const float4*>(base + c_lo) : make_float4(0.f, 0.f, 0.f, 0.f);
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = c_lo + e < C ? base[c_lo + e] : 0.f;
        return make_float4(v[0], v[1], v[2], v[3]);
    };
    auto load_chunk = [&](int c) {
        const int qc = c * kKC;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const int q = qc + s_row + 16 * k;
            const int r = q / U_w, xx = q - r * U_w;              // r = f E_h + y
            ra[k] = load4(dy + ((int64_t)r * E_w + xx) * Cout, o0 + s_col, Cout, q < Q && xx < E_w);
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            int row, col;
            if constexpr (PACKED) {                 // rows of cpt floats, cpt / 4 units each
                const int u = tid + 256 * k;
                row = u / (cpt / 4);
                col = (u - row * (cpt / 4)) * 4;
            } else {
                row = s_row + 16 * k;
                col = i0 + s_col;
            }
            const int q = qc + tw0 + row;
            const int f = q / rowlen;
            const int64_t src = (int64_t)q + (int64_t)f * (fh - 1) * U_w + (int64_t)th * U_w;
            rb[k] = row < rows_b ? load4(x + src * Cin, col, Cin, q < Q) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    auto store_chunk = [&](int buf) {
#pragma unroll
        for (int k = 0; k < 2; ++k)
            *reinterpret_cast<float4*>(lds_a(buf) + (s_row + 16 * k) * kWP + s_col) = ra[k];
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            if constexpr (PACKED) {
                const int u = tid + 256 * k;
                if (u < rows_b * (cpt / 4)) *reinterpret_cast<float4*>(lds_b(buf) + u * 4) = rb[k];
            } else {
                if (s_row + 16 * k < RB) *reinterpret_cast<float4*>(lds_b(buf) + (s_row + 16 * k) * kWP + s_col) = rb[k];
            }
        }
    };

    if (c0 < c1) {
        load_chunk(c0);
        store_chunk(0);
    }
    __syncthreads();
    for (int c = c0; c < c1; ++c) {
        const int buf = (c - c0) & 1;
        const bool more = c + 1 < c1;
        if (more) load_chunk(c + 1);
        const float* A = lds_a(buf) + wm * 32 + l32;
        const float* Bm = lds_b(buf) + wn * 32 + l32;   // packed: column j = wn 32 + l32 of row 0
        const int bstep = PACKED ? cpt : kWP;           // floats between staged rows
        // all TT taps even in a ragged last group (the extra ones are not stored):
        // a tap-dependent branch here would keep a second copy of the accumulators
#pragma unroll 4
        for (int ks = 0; ks < kKC / 2; ++ks) {
            const int p = 2 * ks + half;
            const float av = A[p * kWP];
            bsum += av;
            float bv[TT];
#pragma unroll
            for (int t = 0; t < TT; ++t) bv[t] = PACKED ? Bm[(p + t * g) * bstep] : Bm[(p + t) * kWP];
#pragma unroll
            for (int t = 0; t < TT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv[t], acc[t], 0, 0, 0);
        }
        if (more) store_chunk(buf ^ 1);
        __syncthreads();
    }

    // db[o] = sum_p dy[p][o]: one wave per output-channel half of the workgroups
    // of the first input tile, tap row and tap group adds its two half-wave sums
    bsum += __shfl_xor(bsum, 32);
    if (it == 0 && tg == 0 && th == 0 && wn == 0 && half == 0 && o0 + wm * 32 + l32 < Cout)
        bias_partial[(size_t)split * Cout + o0 + wm * 32 + l32] = bsum;

    // D[i][j] of a 32x32 tile sits in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    const int taps = fh * fw;
    const int jj = wn * 32 + l32;
    const int ii = PACKED ? jj % cpt : i0 + jj;     // input channel of this lane's column
    const int tl = PACKED ? jj / cpt : 0;           // tap of this lane's column within a tile
#pragma unroll
    for (int t = 0; t < TT; ++t) {
        const int k = t * g + tl;                   // tap within the group
        if (k >= ntt) continue;
        float* dst = partial + ((size_t)split * taps + th * fw + tw0 + k) * Cout * Cin;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int o = o0 + wm * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
            if (o < Cout && ii < Cin) dst[(size_t)o * Cin + ii] = acc[t][v];
        }
    }
}

// dW[o][i][th][tw] = sum over splits (in order) of partial[s][tap][o][i], and
// db[o] = sum over splits (in order) of bias_partial[s][o].
__global__ __launch_bounds__(kBT) void wgrad_reduce_kernel(const float* __restrict__ partial,
                                                          const float* __restrict__ bias_partial, int splits,
                                                          int taps, int Cout, int Cin, float* __restrict__ dw,
                                                          float* __restrict__ db) {
    const int64_t n = (int64_t)Cout * Cin * taps;
    const int64_t p = (int64_t)blockIdx.x * kBT + threadIdx.x;
    if (p >= n) {
        const int64_t o = p - n;
        if (o >= Cout) return;
        float s = 0.f;
        for (int k = 0; k < splits; ++k) s += bias_partial[(int64_t)k * Cout + o];
        db[o] = s;
        return;
    }
    const int tap = (int)(p % taps);
    const int64_t oi = p / taps;                 // o * Cin + i
    const int64_t stride = (int64_t)taps * Cout * Cin;
    const float* src = partial + (int64_t)tap * Cout * Cin + oi;
    float s = 0.f;
    for (int k = 0; k < splits; ++k) s += src[k * stride];
    dw[p] = s;                                   // [o][i][th][tw] with tap = th * fw + tw
}

WgradPlan wgrad_plan(int F, int E_h, int E_w, int Cout, int Cin, int fh, int fw) {
    WgradPlan w;
    if (Cin <= kWT / 2) {
        // packed: cpt columns per tap, g taps per tile; at most kMaxPackedTT tiles,
        // the fewest MFMA tiles per row (ntg * tt), then the most taps per group
        w.packed = true;
        w.cpt = 4;
        while (w.cpt < Cin) w.cpt *= 2;
        const int g = kWT / w.cpt;
        int best_work = -1;
        for (int tt = kMaxPackedTT; tt >= 1; --tt) {
            const int ntg = (fw + tt * g - 1) / (tt * g);
            if (best_work < 0 || ntg * tt < best_work) {
                best_work = ntg * tt;
                w.tt = tt;
                w.ntg = ntg;
            }
        }
    } else {
        // the largest group of taps (at most kMaxTT) whose ragged last group wastes
        // at most a tenth of the row's MFMA work
        for (int tt = std::min(fw, kMaxTT); tt >= 1; --tt) {
            const int ntg = (fw + tt - 1) / tt;
            if (10 * (ntg * tt - fw) <= fw) {
                w.tt = tt;
                w.ntg = ntg;
                break;
            }
        }
    }
    w.positions = (int64_t)F * E_h * (E_w + fw - 1);
    w.nchunks = (w.positions + kKC - 1) / kKC;
    w.otiles = (Cout + kWT - 1) / kWT;
    w.itiles = w.packed ? 1 : (Cin + kWT - 1) / kWT;
    const int64_t base = (int64_t)w.otiles * w.itiles * fh * w.ntg;
    // About 512 workgroups run at once (two or three per CU, 53-55 KB of LDS
    // each).  Take at least eight rounds of 512 and, among the split counts up
    // to twice that, the one whose last round is fullest; every split keeps at
    // least 64 chunks, so that a workgroup's prologue and partial-sum stores stay
    // small against its loop (measured on the 512 x 512 frame: 8 -> 64 chunks
    // makes its weight gradients 6.6 -> 5.5 ms).
    const int64_t max_splits = std::max<int64_t>(1, std::min<int64_t>(4096, w.nchunks / 64));
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
    w.bias_partial_floats = (int64_t)w.splits * Cout;
    return w;
}

template <bool VEC, int TT, bool PACKED>
static hipError_t run_wgrad(const float* dy, const float* x, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                            int fh, int fw, const WgradPlan& w, float* partial, float* bpart, hipStream_t s) {
    auto kern = wgrad_mfma_kernel<VEC, TT, PACKED>;
    const size_t lds = wgrad_lds_bytes(TT);
    hipError_t e = allow_dynamic_lds((const void*)kern, lds);
    if (e != hipSuccess) return e;
    const int64_t nblocks = (int64_t)w.otiles * w.itiles * fh * w.ntg * w.splits;
    if (nblocks >= (1ll << 31)) return hipErrorInvalidConfiguration;
    kern<<<dim3((unsigned)nblocks), 256, lds, s>>>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, (int)w.positions,
                                                   (int)w.nchunks, w.otiles, w.itiles, w.ntg, w.splits, w.cpt,
                                                   partial, bpart);
    return hipGetLastError();
}

template <bool VEC>
static hipError_t dispatch_wgrad(const float* dy, const float* x, int E_h, int E_w, int U_h, int U_w, int Cout,
                                 int Cin, int fh, int fw, const WgradPlan& w, float* partial, float* bpart,
                                 hipStream_t s) {
    if (w.packed) {
        switch (w.tt) {
            case 1: return run_wgrad<VEC, 1, true>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
            case 2: return run_wgrad<VEC, 2, true>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
            case 3: return run_wgrad<VEC, 3, true>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
            case 4: return run_wgrad<VEC, 4, true>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        }
        return hipErrorInvalidValue;
    }
    switch (w.tt) {
        case 1: return run_wgrad<VEC, 1, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 2: return run_wgrad<VEC, 2, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 3: return run_wgrad<VEC, 3, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 4: return run_wgrad<VEC, 4, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 5: return run_wgrad<VEC, 5, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 6: return run_wgrad<VEC, 6, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 7: return run_wgrad<VEC, 7, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
        case 8: return run_wgrad<VEC, 8, false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_wgrad(const float* dy, const float* x, int F, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                        int fh, int fw, const WgradPlan& w, float* partial, float* dw, float* db, hipStream_t s) {
    (void)F;
    // positions and chunks are 32-bit in the kernel
    const int span = w.packed ? w.tt * (kWT / w.cpt) : w.tt;   // taps per group
    if (w.positions + span + kKC >= (1ll << 31) || U_w != E_w + fw - 1 || U_h != E_h + fh - 1)
        return hipErrorInvalidConfiguration;
    float* bpart = partial + w.partial_floats;
    const bool vec = Cout % 4 == 0 && Cin % 4 == 0;
    hipError_t e = vec ? dispatch_wgrad<true>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s)
                       : dispatch_wgrad<false>(dy, x, E_h, E_w, U_h, U_w, Cout, Cin, fh, fw, w, partial, bpart, s);
    if (e != hipSuccess) return e;
    const int64_t n = (int64_t)Cout * Cin * fh * fw + Cout;
    wgrad_reduce_kernel<<<dim3((unsigned)ceil_div64(n, kBT)), kBT, 0, s>>>(partial, bpart, w.splits, fh * fw, Cout,
                                                                           Cin, dw, db);
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
