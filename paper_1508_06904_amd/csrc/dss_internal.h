// Internal declarations of the dense-signal-scanning library: the processing
// chain built from the layer list, the per-signal geometry, the plan, and the
// kernel launchers.  Host code only sees these; kernels live in the .hip files.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/dss.h"

namespace dss {

// ------------------------------------------------------------------ errors
void set_error(const char* fmt, ...);
dss_status fail(dss_status s, const char* fmt, ...);
dss_status hip_fail(hipError_t e, const char* what);

// ------------------------------------------------------------------ chain
// One layer of the processing chain (Definition "processing chain", Sect. 4.2):
// a subsignal compatible transformation T_j (a convolution + bias + activation,
// or the identity) followed by a pooling kernel g_j with block size k_j
// (k_j = 1: bypass, end of Sect. 4.2).
struct ChainLayer {
    bool has_conv = false, has_pool = false;
    int c_h = 1, c_w = 1;       // dimensionality reduction constant of T_j
    int k_h = 1, k_w = 1;       // pool block size
    int cin = 0, cout = 0;      // channels entering / leaving the layer
    int act = DSS_ACT_NONE;
    int desc = -1;              // index of the conv descriptor in the caller's list
};

struct Chain {
    int ndim = 2, in_c = 0;
    std::vector<ChainLayer> layers;          // L entries
    int B_h = 1, B_w = 1;                    // receptive field
    std::vector<int> kstar_h, kstar_w;       // k*_0..k*_L
    std::vector<int> u_h, u_w;               // u_0..u_L (Lemma (a))
    int K_h() const { return kstar_h.back(); }
    int K_w() const { return kstar_w.back(); }
    int L() const { return (int)layers.size(); }
    int out_c() const { return layers.empty() ? in_c : layers.back().cout; }
};

dss_status build_chain(const dss_layer* layers, int n, int ndim, int in_c, Chain* out);

// Geometry of one chain layer for a given trimmed/stuffed signal.
struct LayerGeom {
    bool relaxed = false;   // j <= ell: Stride_g (pool with stride k, no Frag), one fragment
    bool dilated = false;   // dilated fashion: one signal, conv and pool taps dil_h x dil_w apart
    int dil_h = 1, dil_w = 1;
    int Uin_h, Uin_w;   // fragment extent entering the layer (U_{j-1})
    int E_h, E_w;       // extent after T_j (U_{j-1} - c_j + 1)
    int U_h, U_w;       // extent after the pooling step (U_j, or W_j for a relaxed layer)
    int Fin_h, Fin_w;   // fragments entering (k*_{j-1} / k*_ell, or 1)
    int Fout_h, Fout_w; // fragments leaving (k*_j / k*_ell, or 1)
};

struct Geom {
    int ell = 0, step_h = 1, step_w = 1;     // mixed level and output sample spacing k*_ell
    int trim_h = 0, trim_w = 0;              // samples trimmed first (trimming mode)
    int H = 0, W = 0, r_h = 0, r_w = 0, D_h = 0, D_w = 0, out_h = 0, out_w = 0;
    std::vector<LayerGeom> L;
    int64_t buf_bytes = 0;      // one ping-pong buffer
    int64_t ws_bytes = 0;       // both buffers
    double conv_flops = 0, pool_bytes = 0, total_bytes = 0;
};

size_t dtype_size(dss_dtype dt);
dss_status compute_geometry(const Chain& ch, dss_dtype dt, int H, int W, int ell, Geom* g);
// EvalStride on a batch of `count` windows: every layer relaxed, Fin_h = count fragments.
dss_status compute_stride_geometry(const Chain& ch, dss_dtype dt, int count, Geom* g);
// EvalDilate on an H x W signal: one fragment, layer j's taps k*_{j-1} apart;
// LayerGeom U = V_j (Lemma "evaldilate" (a)), E = extent after the convolution.
dss_status compute_dilate_geometry(const Chain& ch, dss_dtype dt, int H, int W, Geom* g);

// ------------------------------------------------------------------ plan
enum ConvImpl { CONV_DIRECT = 0, CONV_MFMA_F32 = 1, CONV_MFMA_BF16 = 2 };

struct PlanConv {
    ConvImpl impl = CONV_DIRECT;
    int cin = 0, cout = 0, fh = 1, fw = 1, act = 0;
    int cob = 1, cout_pad = 0;  // direct kernel: outputs per thread, padded Cout
    int bn = 0, cin_pad = 0;    // MFMA kernels: N tile, padded Cin
    void* w = nullptr;          // device weights in the kernel's layout
    float* b = nullptr;         // device bias [cout_pad], zero padded
    // MFMA kernels with the 128-channel N tile also keep the weights packed for the
    // 64-channel tile, used when a launch would leave the GPU short of workgroups
    void* w_alt = nullptr;
    int bn_alt = 0, cout_pad_alt = 0;
    // MFMA convolution followed by a folded 1x1 projection: its weights as
    // [max(cout_pad, cout_pad_alt)][4] binary32 (zero padded), device
    float* w2 = nullptr;
};

// Whether a direct-kernel convolution with Cin input channels runs the lane-sum
// form (conv_direct.hip): few outputs per launch column, filters at most 8 wide,
// input channels a multiple of the wavefront width.  Depends on the layer only,
// so every evaluation fashion sums a layer's outputs in the same order.
inline bool conv_lanesum_ok(int cin, const PlanConv& pc) {
    return cin > 0 && cin % 64 == 0 && pc.cob <= 8 && pc.fw >= 1 && pc.fw <= 8;
}

// The variant a launch over F fragments of Hin x Win (taps dil apart) should use.
PlanConv mfma_launch_variant(const PlanConv& pc, int F, int Hin, int Win, int dil_h, int dil_w, int pad_h = 0,
                             int pad_w = 0);
// How that launch tiles its output: 0 spatial, 1 flat, 2 dilated (dss_launch_record.tile_mode),
// -1 for the direct kernel.
int mfma_tile_mode(const PlanConv& pc, int F, int Hin, int Win, int dil_h, int dil_w, int pad_h = 0, int pad_w = 0);

// Host-side description of a weight-gradient launch (backward.hip).
struct WgradPlan {
    int tt = 1, ntg = 1;         // MFMA tiles per wave (taps, or tap groups when packed), groups per row
    bool packed = false;         // narrow layer: cpt columns per tap, 64 / cpt taps per tile
    int cpt = 64;
    int otiles = 0, itiles = 0, splits = 0;
    int64_t positions = 0;       // F * E_h * U_w: output rows read over the input width
    int64_t nchunks = 0, partial_floats = 0;
    int64_t bias_partial_floats = 0;   // after the weight partial sums in the same buffer
};

struct LaunchRec {
    const char* name;
    int layer;
    double flops, bytes;
    int ev0, ev1;
    int tile_mode;      // dss_launch_record.tile_mode
};

}  // namespace dss

struct dss_plan {
    dss::Chain chain;
    dss_dtype dtype = DSS_F32;
    int device = 0;
    std::vector<dss::PlanConv> convs;     // one per chain layer (impl unused if no conv)
    std::vector<dss::PlanConv> bconvs;    // binary32 plans: the input-gradient convolutions (transposed,
                                          // flipped filters, no bias, no activation)
    // The last chain layer is a 1x1 convolution to at most 4 channels without a
    // pool, after an MFMA convolution without a pool: dense and mixed
    // evaluations fold it into that convolution's epilogue (convs[L-2].w2) and
    // sum the N blocks' partial projections in the final defragmentation.
    bool fuse_proj = false;
    // Sliding max-pool + Frag of one-row fragments in the epilogue of the binary32
    // MFMA convolution before it, or in the direct kernel of a first layer (off
    // with DSS_FUSE_POOL=0 at plan creation).
    bool fuse_pool = true;
    float* proj_b = nullptr;              // device [4]: the projection's bias, zero padded
    int proj_cout = 0, proj_act = 0;
    bool timing = false;
    std::vector<hipEvent_t> events;
    std::vector<dss::LaunchRec> recs;
    // workspace of the evaluations that pass none: allocated on first need,
    // grown to the largest request, freed by dss_plan_destroy
    std::mutex ws_mu;
    void* own_ws = nullptr;
    int64_t own_ws_bytes = 0;
};

namespace dss {

// ------------------------------------------------------------------ evaluation steps (api.cpp)
// Argument checks and geometry of a dense (ell = 0) or mixed evaluation, and
// the plan-device check; nothing is enqueued.
dss_status eval_prepare(dss_plan_t plan, const void* signal, const void* out, int H, int W, int ell, Geom* G);
// The evaluation itself in the workspace ws (at least G.ws_bytes bytes, 256-byte
// aligned).  timed = false records no launch events even with the plan's timing
// on (no event is created).
dss_status eval_run(dss_plan_t plan, const Geom& G, const void* signal, float* out, char* ws, hipStream_t stream,
                    bool timed);

// ------------------------------------------------------------------ kernel launchers
// Element types: binary32 activations are float, bfloat16 activations uint16_t bits.
hipError_t launch_stuff_pack(dss_dtype dt, const void* in, int C, int H, int W, void* out, int D_h,
                             int D_w, hipStream_t s);
// Convolutions over F fragments of Hin x Win; with dil_h x dil_w > 1 (F = 1) the
// taps are dil samples apart (the dilated fashion) and the output has
// Hin - dil_h (fh - 1) x Win - dil_w (fw - 1) samples.
hipError_t launch_conv_direct(dss_dtype tin, dss_dtype tout, const void* in, int F, int Hin, int Win,
                              int dil_h, int dil_w, int Cin, const PlanConv& pc, void* out, hipStream_t s);
// A direct-kernel convolution of F one-row fragments of Win samples (dtype dt in
// and out) with the following sliding max-pool of pool_k (2 to 4) samples and Frag:
// pool_k F fragments of pool_U samples (the convolution's Win - fw + 1 outputs
// must be pool_k pool_U + pool_k - 1).
hipError_t launch_conv_direct_pool(dss_dtype dt, const void* in, int F, int Win, int Cin, const PlanConv& pc,
                                   int pool_k, int pool_U, void* out, hipStream_t s);
hipError_t launch_conv_mfma_f32(const float* in, int F, int Hin, int Win, int dil_h, int dil_w,
                                const PlanConv& pc, float* out, hipStream_t s);
hipError_t launch_conv_mfma_bf16(dss_dtype tout, const uint16_t* in, int F, int Hin, int Win, int dil_h,
                                 int dil_w, const PlanConv& pc, void* out, hipStream_t s);
// As launch_conv_mfma_f32 over fragments with a zero border of pad_h x pad_w
// samples that is not stored (output (Hin + 2 pad_h - fh + 1) x (Win + 2 pad_w - fw + 1)).
hipError_t launch_conv_mfma_f32_padded(const float* in, int F, int Hin, int Win, int pad_h, int pad_w,
                                       const PlanConv& pc, float* out, hipStream_t s);
hipError_t launch_pool_frag(dss_dtype dt, const void* in, int S_h, int S_w, int E_h, int E_w, int C,
                            int k_h, int k_w, void* out, hipStream_t s);
hipError_t launch_patch_pack(dss_dtype dt, const void* in, int C, int H, int W, int O_w, int64_t first, int count,
                             int B_h, int B_w, void* out, hipStream_t s);
hipError_t launch_window_scatter(dss_dtype dt, const void* in, int count, int C, int64_t first, int64_t plane,
                                 float* out, hipStream_t s);
hipError_t launch_pool_dilate(dss_dtype dt, const void* in, int E_h, int E_w, int C, int k_h, int k_w, int dil_h,
                              int dil_w, void* out, hipStream_t s);
hipError_t launch_pool_stride(dss_dtype dt, const void* in, int E_h, int E_w, int C, int k_h, int k_w,
                              void* out, hipStream_t s);
hipError_t launch_defrag_trim(dss_dtype dt, const void* in, int K_h, int K_w, int U_h, int U_w, int C,
                              float* out, int O_h, int O_w, hipStream_t s);
// Defrag + Trim of a folded projection: out = act(bias + sum over nbs channel
// groups of part[g][fragment sample][c]) for c < C <= 4, the groups summed in order.
hipError_t launch_defrag_sum(const float* part, int nbs, int K_h, int K_w, int U_h, int U_w, int C, const float* bias,
                             int act, float* out, int O_h, int O_w, hipStream_t s);
// The same sum for the strided baseline's windows first..first+count-1 (part
// [nbs][count][4]) and for the dilated fashion's last layer (part [nbs][h * w][4]).
hipError_t launch_window_scatter_sum(const float* part, int nbs, int count, int C, const float* bias, int act,
                                     int64_t first, int64_t plane, float* out, hipStream_t s);
hipError_t launch_planar_sum(const float* part, int nbs, int h, int w, int C, const float* bias, int act, float* out,
                             hipStream_t s);
// The binary32 MFMA convolution pc (32- or 64-channel N tile) on fragments of
// one output row, with the sliding max-pool of k samples along the row and
// Frag_k in its epilogue: out is the pool's fragment tensor [k F][1][U][Cout].
hipError_t launch_conv_mfma_pool(const float* in, int F, int Hin, int Win, const PlanConv& pc, int pool_k, float* out,
                                 hipStream_t s);
// The MFMA convolution pc (taps dil apart when dilated) with the folded 1x1
// projection (pc.w2): partial projections [groups][F * Hout * Wout][4] per group
// of 64 channels (32 for the 32-channel N tile) instead of the activations.
hipError_t launch_conv_mfma_proj(const void* in, int F, int Hin, int Win, int dil_h, int dil_w, const PlanConv& pc,
                                 float* part, hipStream_t s);
hipError_t launch_to_planar(dss_dtype dt, const void* in, int F, int h, int w, int C, float* out,
                            hipStream_t s);
hipError_t launch_frag_planar(int elem_bytes, bool inverse, const void* in, int k_h, int k_w, int S_h,
                              int S_w, int C, int H, int W, void* out, hipStream_t s);

// backward (backward.hip)
hipError_t launch_frag_scatter_grad(const float* g, int C, int O_h, int O_w, int K_h, int K_w, int U_h, int U_w,
                                    float* out, hipStream_t s);
hipError_t launch_pool_frag_backward(const float* g, const float* a, int S_h, int S_w, int E_h, int E_w, int C,
                                     int k_h, int k_w, int act, float* out, hipStream_t s);
hipError_t launch_act_backward(const float* g, const float* a, int64_t n, int act, float* out, hipStream_t s);
hipError_t launch_pad_grad(const float* in, int F, int E_h, int E_w, int C, int p_h, int p_w, float* out,
                           hipStream_t s);
WgradPlan wgrad_plan(int F, int E_h, int E_w, int Cout, int Cin, int fh, int fw);
hipError_t launch_wgrad(const float* dy, const float* x, int F, int E_h, int E_w, int U_h, int U_w, int Cout, int Cin,
                        int fh, int fw, const WgradPlan& w, float* partial, float* dw, float* db, hipStream_t s);
hipError_t launch_crop_to_planar(const float* in, int D_w, int C, int H, int W, float* out, hipStream_t s);

// host-side weight packing for the MFMA kernels (conv_mfma.hip)
// Largest dynamic LDS allocation of a workgroup on the current device.
size_t device_lds_limit();
// Lets kern use `bytes` of dynamic LDS on the current device (an opt-in is
// needed above 64 KB; kept per device and kernel).
hipError_t allow_dynamic_lds(const void* kern, size_t bytes);
bool mfma_supports(bool bf16, int fh, int fw);
int mfma_f32_pick_bn(int cout);
int mfma_bf16_pick_bn(int cout);
size_t mfma_f32_packed_floats(const PlanConv& pc);
void mfma_f32_pack(const PlanConv& pc, const float* w_oihw, float* dst);
size_t mfma_bf16_packed_elems(const PlanConv& pc);
void mfma_bf16_pack(const PlanConv& pc, const float* w_oihw, uint16_t* dst);

uint16_t host_f32_to_bf16(float f);

}  // namespace dss
