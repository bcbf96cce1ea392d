// Direct (VALU) convolution over the fragment batch, fused bias + activation.
//
// The multi-channel convolution of Sect. 3.3 applied to every fragment
// independently (Definition "fragmentwise evaluation", Sect. 4.2):
//   out[f][y][x][o] = act( bias[o] + sum_{t_h, t_w, i} w[t_h][t_w][i][o] * in[f][y+t_h][x+t_w][i] )
// for y < Hin - fh + 1, x < Win - fw + 1 (valid convolution, cross-correlation
// tap order).  In the dilated fashion (appendix, Definition "dilate") tap
// (t_h, t_w) reads sample (y + dil_h t_h, x + dil_w t_w) of a single signal.
// Used for the layers that do not suit the MFMA implicit GEMM: the first layer
// (few input channels) and the final projections (few output channels, where
// an MFMA tile of 32 channels would be mostly idle).  Three forms:
//  - conv_direct_kernel: one thread computes COB consecutive output channels of
//    one output sample; the weight reads are uniform across the wavefront and
//    go through the scalar cache (first layers; conv_direct_pool_kernel is its
//    1-D variant with the following sliding max-pool and Frag);
//  - conv_lanesum_kernel: lanes over input channels (a multiple of 64), a
//    butterfly across the lanes per output (few output channels);
//  - conv_narrow_kernel: LDS-staged tiles, one thread per output sample (few
//    output channels, 16 or more input channels not a multiple of 64).
// Accumulation is binary32 (bfloat16 activations are widened).
#include "dev_common.h"
#include "dss_internal.h"

namespace dss {

// COB activated outputs of sample p (channels og .. og + COB - 1), as 16-byte
// vectors where the channel block is whole and aligned.
template <typename Tout, int COB>
__device__ __forceinline__ void store_outputs(Tout* __restrict__ out, int64_t p, int Cout, int og, int act,
                                              const float (&acc)[COB]) {
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
    store_outputs<Tout, COB>(out, p, Cout, og, act, acc);
}

// Few output channels (at most 8) and many input channels (the final
// projections): the plain kernel above reads a whole channel vector per thread,
// so each load instruction touches one cache line per lane.  Here a workgroup
// takes a TH x TW tile of output samples (TH TW = 256, one per thread); per chunk
// of KC input channels the tile's halo of (TH + dil_h (fh - 1)) x
// (TW + dil_w (fw - 1)) samples is read with 16-byte loads into registers (the
// next chunk's loads are issued before this chunk's arithmetic), stored to LDS
// as binary32 with a KC + 4 float pitch (16-byte reads of consecutive samples
// hit disjoint banks), and every thread accumulates its sample from there.  The
// weights of a chunk, taps x KC x COB values read uniformly, go through the
// scalar cache: KC = 32 for 1x1 filters, 16 for wider ones.
constexpr int kNMaxUnits = 8;  // 16-byte staging units per thread and chunk

template <typename Tin, typename Tout, int COB, int KC>
__global__ __launch_bounds__(256) void conv_narrow_kernel(const Tin* __restrict__ in, int Hin, int Win, int Cin,
                                                         const float* __restrict__ w, const float* __restrict__ bias,
                                                         int fh, int fw, int dil_h, int dil_w, int Cout, int CoutP,
                                                         int act, Tout* __restrict__ out, int Hout, int Wout, int TH,
                                                         int TW, int tilesY, int tilesX) {
    constexpr int kNC = KC, kNP = KC + 4;
    constexpr int EPU = 16 / sizeof(Tin);              // channels per 16-byte unit
    constexpr int UPS = kNC / EPU;                     // units per sample and chunk
    extern __shared__ __attribute__((aligned(16))) float sm[];
    const int tiles = tilesY * tilesX;
    const int f = blockIdx.x / tiles, tr = blockIdx.x - f * tiles;
    const int ty0 = (tr / tilesX) * TH, tx0 = (tr % tilesX) * TW;
    const int og = blockIdx.y * COB;
    const int HWd = TW + dil_w * (fw - 1);
    const int nunits = (TH + dil_h * (fh - 1)) * HWd * UPS;
    const int tid = threadIdx.x;
    const int ly = tid / TW, lx = tid - ly * TW;
    const int y = ty0 + ly, x = tx0 + lx;
    const bool active = y < Hout && x < Wout;
    const Tin* in_f = in + (size_t)f * Hin * Win * Cin;
    const bool vec = Cin % EPU == 0;
    float acc[COB];
#pragma unroll
    for (int o = 0; o < COB; ++o) acc[o] = bias[og + o];

    uint4 ru[kNMaxUnits];
    auto load_chunk = [&](int c0) {
#pragma unroll
        for (int k = 0; k < kNMaxUnits; ++k) {
            const int u = tid + 256 * k;
            ru[k] = make_uint4(0u, 0u, 0u, 0u);
            if (u >= nunits) continue;
            const int si = u / UPS, q = u - si * UPS;
            const int hy = si / HWd, hx = si - hy * HWd;
            const int gy = ty0 + hy, gx = tx0 + hx, c = c0 + EPU * q;
            if (gy >= Hin || gx >= Win || c >= Cin) continue;
            const Tin* src = in_f + ((size_t)gy * Win + gx) * Cin + c;
            if (vec) {
                ru[k] = *reinterpret_cast<const uint4*>(src);
            } else {
                Tin t[EPU];
#pragma unroll
                for (int e = 0; e < EPU; ++e) t[e] = c + e < Cin ? src[e] : Tin(0);
                ru[k] = __builtin_bit_cast(uint4, t);
            }
        }
    };
    auto store_chunk = [&]() {
#pragma unroll
        for (int k = 0; k < kNMaxUnits; ++k) {
            const int u = tid + 256 * k;
            if (u >= nunits) continue;
            const int si = u / UPS, q = u - si * UPS;
            float* dst = sm + si * kNP + EPU * q;
            if constexpr (sizeof(Tin) == 4) {
                *reinterpret_cast<uint4*>(dst) = ru[k];
            } else {
                const uint32_t wv[4] = {ru[k].x, ru[k].y, ru[k].z, ru[k].w};
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    *reinterpret_cast<float4*>(dst + 4 * h) = make_float4(
                        __uint_as_float(wv[2 * h] << 16), __uint_as_float(wv[2 * h] & 0xffff0000u),
                        __uint_as_float(wv[2 * h + 1] << 16), __uint_as_float(wv[2 * h + 1] & 0xffff0000u));
            }
        }
    };

    load_chunk(0);
    for (int c0 = 0; c0 < Cin; c0 += kNC) {
        __syncthreads();                               // the previous chunk has been used
        store_chunk();
        __syncthreads();
        if (c0 + kNC < Cin) load_chunk(c0 + kNC);      // in flight during the arithmetic below
        if (!active) continue;
        const int cn = min(kNC, Cin - c0);
        for (int th = 0; th < fh; ++th) {
            for (int tw = 0; tw < fw; ++tw) {
                const float* sp = sm + ((ly + th * dil_h) * HWd + lx + tw * dil_w) * kNP;
                const float* wr = w + ((size_t)(th * fw + tw) * Cin + c0) * CoutP + og;
                if (cn == kNC) {
#pragma unroll
                    for (int q = 0; q < kNC / 4; ++q) {
                        const float4 v4 = *reinterpret_cast<const float4*>(sp + 4 * q);
                        const float v[4] = {v4.x, v4.y, v4.z, v4.w};
#pragma unroll
                        for (int e = 0; e < 4; ++e)
#pragma unroll
                            for (int o = 0; o < COB; ++o) acc[o] = fmaf(v[e], wr[(4 * q + e) * CoutP + o], acc[o]);
                    }
                } else {
                    for (int c = 0; c < cn; ++c)
#pragma unroll
                        for (int o = 0; o < COB; ++o) acc[o] = fmaf(sp[c], wr[c * CoutP + o], acc[o]);
                }
            }
        }
    }
    if (active) store_outputs<Tout, COB>(out, ((int64_t)f * Hout + y) * Wout + x, Cout, og, act, acc);
}

// Few output channels and input channels a multiple of 64 (the lane-sum form).
// A wavefront computes P = 64 / COB output samples of one row, consecutive or,
// in the dilated fashion, dil_w apart (one phase of the row), for COB output
// channels; lane c owns the input channels c, c + 64, ...  Per filter row and
// channel group it loads the P + FW - 1 input samples of its channel that the
// P outputs touch (one 256-byte load per sample across the wavefront, binary32)
// and its FW x COB weights, and accumulates P x COB partial sums over its own
// channels: no LDS and no scalar loads in the loop.  A butterfly across the
// lanes then adds up the 64 partial sums of each output: at each of six steps a
// lane keeps half of its values, sends the other half to the lane whose index
// differs in one bit and adds what it receives, so lane l ends with output
// value l (sample l / COB, channel l % COB), which it stores with bias and
// activation.  An output's sum has the same order wherever its tile lies, so
// the dense, strided, mixed and dilated fashions agree bit for bit.
template <int N>
__device__ __forceinline__ void lane_reduce_scatter(float (&v)[64], int lane) {
    // v[0 .. 2N) -> v[0 .. N): lanes with bit N set keep the upper half
    if constexpr (N >= 16) {
        // across rows of 16 lanes: swap the upper half-wave (N = 32) or the odd
        // rows (N = 16) of the lower values with the lower half-wave or the even
        // rows of the upper values; each lane then holds its own and its
        // partner's copy of the value it keeps
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const uint32_t a = __float_as_uint(v[i]), b = __float_as_uint(v[i + N]);
            const auto r = N == 32 ? __builtin_amdgcn_permlane32_swap(a, b, false, false)
                                   : __builtin_amdgcn_permlane16_swap(a, b, false, false);
            v[i] = __uint_as_float(r[0]) + __uint_as_float(r[1]);
        }
    } else {
        // within a row: the lower lanes of each pair read lane + N, the upper
        // ones lane - N (row shifts of the data-parallel primitives)
        const bool upper = (lane & N) != 0;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const uint32_t a = __float_as_uint(v[i]), b = __float_as_uint(v[i + N]);
            const float lo = v[i] + __uint_as_float(__builtin_amdgcn_update_dpp(0u, a, 0x100 + N, 0xf, 0xf, false));
            const float hi = v[i + N] + __uint_as_float(__builtin_amdgcn_update_dpp(0u, b, 0x110 + N, 0xf, 0xf, false));
            v[i] = upper ? hi : lo;
        }
    }
    if constexpr (N > 1) lane_reduce_scatter<N / 2>(v, lane);
}

// Word 3 of a raw buffer resource on gfx9-family GPUs (32-bit data format).
constexpr int kBufferWord3 = 0x00020000;

template <typename Tin, typename Tout, int COB, int FW, bool ONE_STEP>
__global__ __launch_bounds__(256) void conv_lanesum_kernel(const Tin* __restrict__ in, int Hin, int Win, int Cin,
                                                          const float* __restrict__ w, const float* __restrict__ bias,
                                                          int fh, int dil_h, int dil_w, int Cout, int CoutP, int act,
                                                          Tout* __restrict__ out, int Hout, int Wout, int tiles_row,
                                                          int64_t ntiles) {
    constexpr int P = 64 / COB;
    constexpr int NW = P + FW - 1;                    // input samples per row of taps
    const int lane = threadIdx.x & 63;
    // A wavefront takes the tiles wave, wave + nwaves, ...; per tile the steps
    // (filter row, channel group).  Loads run ahead of the arithmetic in
    // rotating register sets: with one step per tile (ONE_STEP: one filter row,
    // 64 input channels, at least two output channels) the weights stay in
    // registers and the samples load two tiles ahead, otherwise samples and
    // weights load one step ahead.  Tiles
    // and addresses but the lane's channel offset are uniform: scalar registers.
    const int64_t nwaves = (int64_t)gridDim.x * 4;
    int64_t tile = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (tile >= ntiles) return;
    const int og = blockIdx.y * COB;
    const int groups = Cin / 64, steps = fh * groups;

    auto fetch_samples = [&](int64_t tl, int st, float (&win)[NW]) {
        const int64_t fr = tl / tiles_row;            // fragment * Hout + output row
        const int t = (int)(tl - fr * tiles_row);
        const int x0 = t % dil_w + (t / dil_w) * P * dil_w;
        const int th = st / groups, c0 = (st - th * groups) * 64;
        const int64_t f = fr / Hout;
        const int y = (int)(fr - f * Hout);
        // the row as a buffer: the sample offset goes in a scalar register, the
        // lane's channel offset in a vector register, so a load costs no vector
        // address arithmetic
        const Tin* row = in + ((f * Hin + y + th * dil_h) * (int64_t)Win) * Cin + c0;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void*)row, 0, (int)(((int64_t)Win * Cin - c0) * (int64_t)sizeof(Tin)), kBufferWord3);
        const int voff = lane * (int)sizeof(Tin);
        auto sample = [&](int xs) {
            // past the row end: the last sample (its outputs are past the end too)
            const int soff = min(xs, Win - 1) * Cin * (int)sizeof(Tin);
            if constexpr (sizeof(Tin) == 4)
                return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, 0));
            else
                return bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rs, voff, soff, 0));
        };
        if (x0 + (NW - 1) * dil_w < Win) {            // the whole window lies in the row
#pragma unroll
            for (int i = 0; i < NW; ++i) win[i] = sample(x0 + i * dil_w);
        } else {
#pragma unroll
            for (int i = 0; i < NW; ++i) {
                const int xs = x0 + i * dil_w;
                const float v = sample(xs);
                win[i] = xs < Win ? v : 0.f;
            }
        }
    };
    auto fetch_weights = [&](int st, float (&wv)[FW][COB]) {
        const int th = st / groups, c0 = (st - th * groups) * 64;
        const float* wrow = w + ((int64_t)th * FW * Cin + c0) * CoutP + og;
#pragma unroll
        for (int tw = 0; tw < FW; ++tw)
#pragma unroll
            for (int o = 0; o < COB; ++o) wv[tw][o] = (wrow + (int64_t)tw * Cin * CoutP)[lane * CoutP + o];
    };

    float acc[64];
#pragma unroll
    for (int v = 0; v < 64; ++v) acc[v] = 0.f;
    auto accumulate = [&](const float (&win)[NW], const float (&wv)[FW][COB]) {
#pragma unroll
        for (int tw = 0; tw < FW; ++tw)
#pragma unroll
            for (int p = 0; p < P; ++p)
#pragma unroll
                for (int o = 0; o < COB; ++o) acc[p * COB + o] = fmaf(win[p + tw], wv[tw][o], acc[p * COB + o]);
    };
    // the tile is complete: sum across the lanes, store, clear
    auto finish = [&]() {
        lane_reduce_scatter<32>(acc, lane);
        const int64_t fr = tile / tiles_row;
        const int t = (int)(tile - fr * tiles_row);
        const int p = lane / COB, o = lane - (lane / COB) * COB;
        const int x = t % dil_w + (t / dil_w) * P * dil_w + p * dil_w;
        if (x < Wout && og + o < Cout)
            store_elem(out + (fr * Wout + x) * Cout + og + o, activate(act, acc[0] + bias[og + o]));
#pragma unroll
        for (int v = 0; v < 64; ++v) acc[v] = 0.f;
    };

    if constexpr (ONE_STEP) {
        float wv[FW][COB];
        fetch_weights(0, wv);
        // tile on `win` while the tile two ahead loads into `nwin`; false when
        // no tile is left
        auto step = [&](const float (&win)[NW], float (&nwin)[NW]) {
            const int64_t ahead = tile + 2 * nwaves;
            if (ahead < ntiles) fetch_samples(ahead, 0, nwin);
            accumulate(win, wv);
            finish();
            tile += nwaves;
            return tile < ntiles;
        };
        float winA[NW], winB[NW], winC[NW];
        fetch_samples(tile, 0, winA);
        if (tile + nwaves < ntiles) fetch_samples(tile + nwaves, 0, winB);
        while (step(winA, winC) && step(winB, winA) && step(winC, winB)) {
        }
    } else {
        int st = 0;
        // one step on (win, wv) with the next step's loads into (nwin, nwv);
        // false when no step is left
        auto step = [&](const float (&win)[NW], const float (&wv)[FW][COB], float (&nwin)[NW],
                        float (&nwv)[FW][COB]) {
            int64_t ntile = tile;
            int nst = st + 1;
            if (nst == steps) {
                nst = 0;
                ntile += nwaves;
            }
            const bool more = ntile < ntiles;
            if (more) {
                fetch_samples(ntile, nst, nwin);
                fetch_weights(nst, nwv);
            }
            accumulate(win, wv);
            if (nst == 0) finish();
            tile = ntile;
            st = nst;
            return more;
        };
        float winA[NW], winB[NW], wvA[FW][COB], wvB[FW][COB];
        fetch_samples(tile, 0, winA);
        fetch_weights(0, wvA);
        while (step(winA, wvA, winB, wvB) && step(winB, wvB, winA, wvA)) {
        }
    }
}

template <typename Tin, typename Tout, int COB, int FW, bool ONE_STEP>
static void launch_lanesum(const void* in, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc, void* out,
                           int Hout, int Wout, int tiles_row, int64_t ntiles, hipStream_t s) {
    // as many workgroups as the GPU holds at once, each wavefront looping over
    // its tiles
    static const int64_t resident = [] {
        int per_cu = 0, dev = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, conv_lanesum_kernel<Tin, Tout, COB, FW, ONE_STEP>,
                                                         256, 0) != hipSuccess ||
            per_cu < 1)
            per_cu = 2;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 256;
        return (int64_t)per_cu * cus;
    }();
    const int64_t wgs = std::min<int64_t>(ceil_div64(ntiles, 4), resident);
    const dim3 grid((unsigned)wgs, (unsigned)(pc.cout_pad / COB));
    conv_lanesum_kernel<Tin, Tout, COB, FW, ONE_STEP><<<grid, 256, 0, s>>>(
        (const Tin*)in, Hin, Win, Cin, (const float*)pc.w, pc.b, pc.fh, dh, dw, pc.cout, pc.cout_pad, pc.act,
        (Tout*)out, Hout, Wout, tiles_row, ntiles);
}

template <typename Tin, typename Tout, int COB, int FW>
static void run_lanesum(const void* in, int F, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc,
                        void* out, int Hout, int Wout, hipStream_t s) {
    constexpr int P = 64 / COB;
    const int64_t blocks = ceil_div64(ceil_div64(Wout, dw), P);     // per phase of a row
    const int tiles_row = (int)(blocks * dw);
    const int64_t ntiles = (int64_t)F * Hout * tiles_row;
    // three sample windows of up to 32 + 7 samples fit beside the accumulators
    if constexpr (COB >= 2) {
        if (pc.fh == 1 && Cin == 64) {
            launch_lanesum<Tin, Tout, COB, FW, true>(in, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, tiles_row, ntiles,
                                                     s);
            return;
        }
    }
    launch_lanesum<Tin, Tout, COB, FW, false>(in, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, tiles_row, ntiles, s);
}

template <typename Tin, typename Tout, int COB>
static void dispatch_lanesum(const void* in, int F, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc,
                             void* out, int Hout, int Wout, hipStream_t s) {
    switch (pc.fw) {
        case 1: run_lanesum<Tin, Tout, COB, 1>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 2: run_lanesum<Tin, Tout, COB, 2>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 3: run_lanesum<Tin, Tout, COB, 3>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 4: run_lanesum<Tin, Tout, COB, 4>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 5: run_lanesum<Tin, Tout, COB, 5>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 6: run_lanesum<Tin, Tout, COB, 6>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        case 7: run_lanesum<Tin, Tout, COB, 7>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
        default: run_lanesum<Tin, Tout, COB, 8>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s); break;
    }
}

// Tile of the narrow kernel: the width (16 .. 256, a power of two) that computes
// the fewest masked samples among those whose halo fits 64 KB of LDS and the
// staging registers; TH = 0 if none does.
static void narrow_tile(int Hout, int Wout, int fh, int fw, int dh, int dw, int kc, int units_per_sample, int& TH,
                        int& TW, size_t& lds) {
    TH = TW = 0;
    int64_t best = -1;
    for (int tw = 16; tw <= 256; tw *= 2) {
        const int th = 256 / tw;
        const int64_t samples = (int64_t)(th + dh * (fh - 1)) * (tw + dw * (fw - 1));
        const size_t l = (size_t)samples * (kc + 4) * sizeof(float);
        if (l > 64 * 1024 || samples * units_per_sample > 256 * kNMaxUnits) continue;
        const int64_t work = ceil_div64(Hout, th) * th * ceil_div64(Wout, tw) * tw;
        if (best < 0 || work < best) {
            best = work;
            TH = th;
            TW = tw;
            lds = l;
        }
    }
}

template <typename Tin, typename Tout, int COB>
static void run_direct(const void* in, int F, int Hin, int Win, int dh, int dw, int Cin, const PlanConv& pc, void* out,
                       hipStream_t s) {
    const int Hout = Hin - dh * (pc.fh - 1), Wout = Win - dw * (pc.fw - 1);
    if constexpr (COB <= 8) {
        if (conv_lanesum_ok(Cin, pc)) {
            dispatch_lanesum<Tin, Tout, COB>(in, F, Hin, Win, dh, dw, Cin, pc, out, Hout, Wout, s);
            return;
        }
    }
    const int kc = pc.fh * pc.fw == 1 ? 32 : 16;
    if (Cin >= 16 && pc.cout_pad <= 8) {
        int TH, TW;
        size_t lds = 0;
        narrow_tile(Hout, Wout, pc.fh, pc.fw, dh, dw, kc, kc / (16 / (int)sizeof(Tin)), TH, TW, lds);
        const int tilesY = (int)ceil_div64(Hout, TH > 0 ? TH : 1), tilesX = (int)ceil_div64(Wout, TW > 0 ? TW : 1);
        if (TH > 0 && (int64_t)F * tilesY * tilesX < (1ll << 31)) {
            const dim3 grid((unsigned)((int64_t)F * tilesY * tilesX), (unsigned)(pc.cout_pad / COB));
            auto kern = kc == 32 ? conv_narrow_kernel<Tin, Tout, COB, 32> : conv_narrow_kernel<Tin, Tout, COB, 16>;
            kern<<<grid, 256, lds, s>>>((const Tin*)in, Hin, Win, Cin, (const float*)pc.w, pc.b, pc.fh, pc.fw, dh, dw,
                                        pc.cout, pc.cout_pad, pc.act, (Tout*)out, Hout, Wout, TH, TW, tilesY, tilesX);
            return;
        }
    }
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

// A direct-kernel convolution of one-row fragments with the following sliding
// max-pool of k samples along the row and Frag_k (EvalSlide_j = Frag_k o
// Slide_k o T_j of Definition "processing chain", one launch): a thread takes
// pooled position x of fragment f and COB output channels, computes the k
// activated convolution outputs x .. x + k - 1 (each summed in the same order
// as conv_direct_kernel, from the bias over taps and channels) and writes
// their maximum to sample x div k of fragment (x mod k) F + f (Lemma
// "frag-ops" along the row).  The unpooled activations are never stored.
template <typename Tin, typename Tout, int COB, int KP>
__global__ __launch_bounds__(256) void conv_direct_pool_kernel(const Tin* __restrict__ in, int Win, int Cin,
                                                              const float* __restrict__ w,
                                                              const float* __restrict__ bias, int fw, int Cout,
                                                              int CoutP, int act, int pool_U, int F,
                                                              Tout* __restrict__ out, int64_t npos) {
    // KP = k: the k outputs accumulate side by side, each weight read once per thread
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (p >= npos) return;
    const int og = blockIdx.y * COB;
    const int row = KP * pool_U;                       // pooled positions per fragment (before Frag)
    const int64_t f = p / row;
    const int x = (int)(p - f * row);
    const Tin* base = in + (f * Win + x) * Cin;
    float acc[KP][COB];
#pragma unroll
    for (int t = 0; t < KP; ++t)
#pragma unroll
        for (int o = 0; o < COB; ++o) acc[t][o] = bias[og + o];
    for (int tw = 0; tw < fw; ++tw) {
        const float* wr = w + (int64_t)tw * Cin * CoutP + og;
        for (int i = 0; i < Cin; ++i) {
            float wv[COB];
#pragma unroll
            for (int o = 0; o < COB; ++o) wv[o] = wr[(int64_t)i * CoutP + o];
#pragma unroll
            for (int t = 0; t < KP; ++t) {
                const float v = to_f32(base[(int64_t)(t + tw) * Cin + i]);
#pragma unroll
                for (int o = 0; o < COB; ++o) acc[t][o] = fmaf(v, wv[o], acc[t][o]);
            }
        }
    }
    float mx[COB];
#pragma unroll
    for (int o = 0; o < COB; ++o) {
        mx[o] = activate(act, acc[0][o]);
#pragma unroll
        for (int t = 1; t < KP; ++t) mx[o] = fmaxf(mx[o], activate(act, acc[t][o]));
    }
    const int64_t fo = (int64_t)(x % KP) * F + f;
    store_outputs<Tout, COB>(out, fo * pool_U + x / KP, Cout, og, 0, mx);
}

template <typename Tin, typename Tout, int KP>
static void dispatch_direct_pool(const void* in, int F, int Win, int Cin, const PlanConv& pc, int pool_U, void* out,
                                 hipStream_t s) {
    const int64_t npos = (int64_t)F * KP * pool_U;
    const dim3 grid((unsigned)ceil_div64(npos, 256), (unsigned)(pc.cout_pad / pc.cob));
#define DSS_DIRECT_POOL(C)                                                                                            \
    conv_direct_pool_kernel<Tin, Tout, C, KP><<<grid, 256, 0, s>>>((const Tin*)in, Win, Cin, (const float*)pc.w, pc.b, \
                                                                   pc.fw, pc.cout, pc.cout_pad, pc.act, pool_U, F,      \
                                                                   (Tout*)out, npos)
    switch (pc.cob) {
        case 16: DSS_DIRECT_POOL(16); break;
        case 8: DSS_DIRECT_POOL(8); break;
        case 4: DSS_DIRECT_POOL(4); break;
        case 2: DSS_DIRECT_POOL(2); break;
        default: DSS_DIRECT_POOL(1); break;
    }
#undef DSS_DIRECT_POOL
}

template <typename Tin, typename Tout>
static hipError_t dispatch_pool_k(const void* in, int F, int Win, int Cin, const PlanConv& pc, int pool_k, int pool_U,
                                  void* out, hipStream_t s) {
    switch (pool_k) {
        case 2: dispatch_direct_pool<Tin, Tout, 2>(in, F, Win, Cin, pc, pool_U, out, s); break;
        case 3: dispatch_direct_pool<Tin, Tout, 3>(in, F, Win, Cin, pc, pool_U, out, s); break;
        case 4: dispatch_direct_pool<Tin, Tout, 4>(in, F, Win, Cin, pc, pool_U, out, s); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_conv_direct_pool(dss_dtype dt, const void* in, int F, int Win, int Cin, const PlanConv& pc,
                                   int pool_k, int pool_U, void* out, hipStream_t s) {
    if (pc.fh != 1 || pool_k < 2 || pool_k > 4 || (Win - pc.fw + 1) - pool_k + 1 != pool_k * pool_U)
        return hipErrorInvalidValue;
    if (F <= 0 || pool_U <= 0) return hipSuccess;
    if (dt == DSS_F32) return dispatch_pool_k<float, float>(in, F, Win, Cin, pc, pool_k, pool_U, out, s);
    return dispatch_pool_k<uint16_t, uint16_t>(in, F, Win, Cin, pc, pool_k, pool_U, out, s);
}

hipError_t launch_conv_direct(dss_dtype tin, dss_dtype tout, const void* in, int F, int Hin, int Win, int dil_h,
                              int dil_w, int Cin, const PlanConv& pc, void* out, hipStream_t s) {
    // the lane-sum form addresses a row as a buffer of at most 2^31 bytes
    if (conv_lanesum_ok(Cin, pc) && (int64_t)Win * Cin * (tin == DSS_F32 ? 4 : 2) > INT32_MAX)
        return hipErrorInvalidValue;
    if (tin == DSS_F32)
        dispatch_cob<float, float>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    else if (tout == DSS_F32)
        dispatch_cob<uint16_t, float>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    else
        dispatch_cob<uint16_t, uint16_t>(in, F, Hin, Win, dil_h, dil_w, Cin, pc, out, s);
    return hipGetLastError();
}

}  // namespace dss
