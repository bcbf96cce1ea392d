// Direct (VALU) convolution over the fragment batch, fused bias + activation.
//
// The multi-channel convolution of Sect. 3.3 applied to every fragment
// independently (Definition "fragmentwise evaluation", Sect. 4.2):
//   out[f][y][x][o] = act( bias[o] + sum_{t_h, t_w, i} w[t_h][t_w][i][o] * in[f][y+t_h][x+t_w][i] )
// for y < Hin - fh + 1, x < Win - fw + 1 (valid convolution, cross-correlation
// tap order).  In the dilated fashion (appendix, Definition "dilate") tap
// (t_h, t_w) reads sample (y + dil_h t_h, x + dil_w t_w) of a single signal.
// Used for the layers that do not suit the MFMA implicit GEMM: the first layer
// (few input channels) and the final projections (few output channels).  One thread computes COB consecutive output channels of one output
// sample; the weight reads are uniform across the wavefront and go through the
// scalar cache.  Accumulation is binary32 (bfloat16 activations are widened).
#include "dev_common.h"
#include "dss_internal.h"

namespace dss {

template <typename Tin, typename Tout, int COB, int VEC>
__global__ __launch_bounds__(256) void conv_direct_kernel(const Tin* __restrict__ in, int Hin, int Win, int Cin,
                                                         const float* __restrict__ w, const float* __restrict__ bias,
                                                         int fh, int fw, int dil_h, int dil_w, int Cout,
                                                         int CoutP, int act, Tout* __restrict__ out, int Hout,
                                                         int Wout, int64_t npix) {
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (p >= npix) return;
    const int og = blockIdx.y * COB;
    const int x = (int)(p % Wout);
    const int64_t t = p / Wout;
    const int y = (int)(t % Hout);
    const int64_t f = t / Hout;
    const Tin* base = in + ((f * Hin + y) * Win + x) * Cin;
    float acc[COB];
#pragma unroll
    for (int o = 0; o < COB; ++o) acc[o] = bias[og + o];
    for (int th = 0; th < fh; ++th) {
        for (int tw = 0; tw < fw; ++tw) {
            const Tin* px = base + ((int64_t)th * dil_h * Win + (int64_t)tw * dil_w) * Cin;
            const float* wr = w + (int64_t)((th * fw + tw) * Cin) * CoutP + og;
            for (int i = 0; i < Cin; i += VEC) {
                float v[VEC];
                VecIO<Tin, VEC>::load(px + i, v);
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
#pragma unroll
                    for (int o = 0; o < COB; ++o) acc[o] = fmaf(v[e], wr[(int64_t)(i + e) * CoutP + o], acc[o]);
                }
            }
        }
    }
    Tout* op = out + p * Cout + og;
    const bool aligned16 = ((uintptr_t)out & 15) == 0;
    if constexpr (sizeof(Tout) == 4 && COB % 4 == 0) {
        if (aligned16 && Cout % 4 == 0 && og + COB <= Cout) {   // 16-byte aligned: full vectors
#pragma unroll
            for (int o = 0; o < COB; o += 4)
                *reinterpret_cast<float4*>(op + o) = make_float4(activate(act, acc[o]), activate(act, acc[o + 1]),
                                                                 activate(act, acc[o + 2]), activate(act, acc[o + 3]));
            return;
        }
    }
    if constexpr (sizeof(Tout) == 2 && COB % 8 == 0) {
        if (aligned16 && Cout % 8 == 0 && og + COB <= Cout) {   // 8 bfloat16 channels per 16-byte store
#pragma unroll
            for (int o = 0; o < COB; o += 8) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[e] = (uint32_t)f32_to_bf16(activate(act, acc[o + 2 * e])) |
                           ((uint32_t)f32_to_bf16(activate(act, acc[o + 2 * e + 1])) << 16);
                *reinterpret_cast<uint4*>(op + o) = make_uint4(w[0], w[1], w[2], w[3]);
            }
            return;
        }
    }
#pragma unroll
    for (int o = 0; o < COB; ++o)
        if (og + o < Cout) store_elem(op + o, activate(act, acc[o]));
}

template <typename Tin, typename Tout, int COB>
static void run_direct(const void* in, int F, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc, void* out,
                       hipStream_t s) {
    const int Hout = Hin - dh * (pc.fh - 1), Wout = Win - dw * (pc.fw - 1);
    const int64_t npix = (int64_t)F * Hout * Wout;
    const dim3 grid((unsigned)ceil_div64(npix, 256), (unsigned)(pc.cout_pad / COB));
    const int vec_ok = (Cin % 4 == 0);
    if (vec_ok)
        conv_direct_kernel<Tin, Tout, COB, 4><<<grid, 256, 0, s>>>((const Tin*)in, Hin, Win, Cin, (const float*)pc.w,
                                                                   pc.b, pc.fh, pc.fw, dh, dw, pc.cout, pc.cout_pad, pc.act,
                                                                   (Tout*)out, Hout, Wout, npix);
    else
        conv_direct_kernel<Tin, Tout, COB, 1><<<grid, 256, 0, s>>>((const Tin*)in, Hin, Win, Cin, (const float*)pc.w,
                                                                   pc.b, pc.fh, pc.fw, dh, dw, pc.cout, pc.cout_pad, pc.act,
                                                                   (Tout*)out, Hout, Wout, npix);
}

template <typename Tin, typename Tout>
static void dispatch_cob(const void* in, int F, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc,
                         void* out, hipStream_t s) {
    switch (pc.cob) {
        case 16: run_direct<Tin, Tout, 16>(in, F, Hin, Win, dh, dw, Cin, pc, out, s); break;
        case 8: run_direct<Tin, Tout, 8>(in, F, Hin, Win, dh, dw, Cin, pc, out, s); break;
        case 4: run_direct<Tin, Tout, 4>(in, F, Hin, Win, dh, dw, Cin, pc, out, s); break;
        case 2: run_direct<Tin, Tout, 2>(in, F, Hin, Win, dh, dw, Cin, pc, out, s); break;
        default: run_direct<Tin, Tout, 1>(in, F, Hin, Win, dh, dw, Cin, pc, out, s); break;
    }
}

hipError_t launch_conv_direct(dss_dtype tin, dss_dtype tout, const void* in, int F, int Hin, int Win, int dil_h,
                              int dil_w, int Cin, const PlanConv& pc, void* out, hipStream_t s) {
    if (tin == DSS_F32)
        dispatch_cob<float, float>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    else if (tout == DSS_F32)
        dispatch_cob<uint16_t, float>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    else
        dispatch_cob<uint16_t, uint16_t>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    return hipGetLastError();
}

}  // namespace dss
