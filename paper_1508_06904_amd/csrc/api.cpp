// C ABI of the dense-signal-scanning library: argument validation, plans,
// the launch sequence of the dense evaluation, Frag/Defrag entry points and
// launch telemetry.
//
// Dense evaluation (Theorem "processing chain", Sect. 4.3):
//   Stuff_r  ->  for j = 1..L: [conv T_j]  [sliding max-pool + Frag_{k_j}]  ->  Defrag_{k*_L} + Trim_r
// Dilated evaluation (appendix, Definition "evaldilate"):
//   pack  ->  for j = 1..L: [conv with taps k*_{j-1} apart] [max with taps k*_{j-1} apart]  ->  planar
// Mixed evaluation at level ell (appendix, Theorem "evalrelaxslide"):
//   Trim or Stuff  ->  for j <= ell: [conv T_j] [max-pool with stride k_j]
//                  ->  for j > ell:  [conv T_j] [sliding max-pool + Frag_{k_j}]
//                  ->  Defrag_{k*_L / k*_ell} + trim to the output extent
// Every intermediate stays in one of two ping-pong halves of the caller's
// workspace, in the channels-last fragment layout [F][h][w][C] (fragment index
// linearised row-major over (row fragment, column fragment)).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>

#include "dss_internal.h"

namespace dss {

static thread_local std::string g_err;

void set_error(const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
}

dss_status fail(dss_status s, const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

dss_status hip_fail(hipError_t e, const char* what) {
    g_err = std::string(what) + ": " + hipGetErrorName(e) + " (" + hipGetErrorString(e) + ")";
    return e == hipErrorOutOfMemory ? DSS_E_NOMEM : DSS_E_HIP;
}

uint16_t host_f32_to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);                                           // round to nearest even
    return (uint16_t)(u >> 16);
}

// Kernel choice per convolution.  The MFMA implicit GEMM wants a contraction
// deep enough to fill its K loop (at least 16 input channels, channel rows of
// whole 16-byte units); the first layers with few input channels go to the
// direct VALU kernel.  Narrow outputs (the final projections) still use MFMA
// with the 32-channel N tile: the padded output channels cost MFMA cycles the
// layer has to spare, while the direct kernel would be limited by its
// uncoalesced reads of the wide input rows.
static ConvImpl choose_impl(int cin, int cout, int fh, int fw, dss_dtype dt) {
    // Tuning / cross-check override: DSS_CONV_KERNEL=direct selects the VALU
    // kernel for every convolution of plans created afterwards.
    const char* force = getenv("DSS_CONV_KERNEL");
    if (force && std::strcmp(force, "direct") == 0) return CONV_DIRECT;
    // few input channels (first layers), or few output channels in binary32
    // (final projections, where a 32-channel MFMA tile would be mostly idle; the
    // LDS-staged direct kernel streams them faster; with bfloat16 inputs the
    // MFMA tile still wins)
    if (cin < 16 || (cout <= 8 && dt == DSS_F32)) return CONV_DIRECT;
    if (dt == DSS_F32 && cin % 4 == 0 && mfma_supports(false, fh, fw)) return CONV_MFMA_F32;
    if (dt == DSS_BF16 && cin % 8 == 0 && mfma_supports(true, fh, fw)) return CONV_MFMA_BF16;
    return CONV_DIRECT;
}

// Packs one convolution (weights [cout][cin][fh][fw] binary32, cross-correlation
// order; bias [cout] or NULL) into the layout of the kernel chosen for it and
// copies it to the current device.
static dss_status upload_conv(int cin, int cout, int fh, int fw, int act, const float* weight, const float* bias_in,
                              dss_dtype dtype, PlanConv& pc) {
    pc.cin = cin;
    pc.cout = cout;
    pc.fh = fh;
    pc.fw = fw;
    pc.act = act;
    pc.impl = choose_impl(cin, cout, fh, fw, dtype);
    const bool bf16 = dtype == DSS_BF16;
    std::vector<float> bias;
    std::vector<char> wbuf;
    size_t wbytes = 0;
    if (pc.impl == CONV_DIRECT) {
        // [fh][fw][cin][cout_pad] binary32 (bfloat16-rounded values for bfloat16 plans)
        pc.cob = cout >= 16 ? 16 : cout >= 8 ? 8 : cout >= 4 ? 4 : cout >= 2 ? 2 : 1;
        pc.cout_pad = (cout + pc.cob - 1) / pc.cob * pc.cob;
        wbytes = sizeof(float) * (size_t)fh * fw * cin * pc.cout_pad;
        wbuf.assign(wbytes, 0);
        float* w = reinterpret_cast<float*>(wbuf.data());
        for (int o = 0; o < cout; ++o)
            for (int i = 0; i < cin; ++i)
                for (int th = 0; th < fh; ++th)
                    for (int tw = 0; tw < fw; ++tw) {
                        float v = weight[(((size_t)o * cin + i) * fh + th) * fw + tw];
                        if (bf16) {
                            const uint32_t u = (uint32_t)host_f32_to_bf16(v) << 16;
                            std::memcpy(&v, &u, 4);
                        }
                        w[(((size_t)th * fw + tw) * cin + i) * pc.cout_pad + o] = v;
                    }
    } else if (pc.impl == CONV_MFMA_F32) {
        pc.bn = mfma_f32_pick_bn(cout);
        pc.cin_pad = (cin + 15) / 16 * 16;
        pc.cout_pad = (cout + pc.bn - 1) / pc.bn * pc.bn;
        wbytes = sizeof(float) * mfma_f32_packed_floats(pc);
        wbuf.assign(wbytes, 0);
        mfma_f32_pack(pc, weight, reinterpret_cast<float*>(wbuf.data()));
    } else {
        pc.bn = mfma_bf16_pick_bn(cout);
        pc.cin_pad = (cin + 31) / 32 * 32;
        pc.cout_pad = (cout + pc.bn - 1) / pc.bn * pc.bn;
        wbytes = sizeof(uint16_t) * mfma_bf16_packed_elems(pc);
        wbuf.assign(wbytes, 0);
        mfma_bf16_pack(pc, weight, reinterpret_cast<uint16_t*>(wbuf.data()));
    }
    // the 64-channel tile's packing, for launches too small for the 128-channel one
    std::vector<char> abuf;
    if (pc.impl != CONV_DIRECT && pc.bn == 128) {
        PlanConv alt = pc;
        alt.bn = 64;
        alt.cout_pad = (cout + 63) / 64 * 64;
        pc.bn_alt = alt.bn;
        pc.cout_pad_alt = alt.cout_pad;
        if (pc.impl == CONV_MFMA_F32) {
            abuf.assign(sizeof(float) * mfma_f32_packed_floats(alt), 0);
            mfma_f32_pack(alt, weight, reinterpret_cast<float*>(abuf.data()));
        } else {
            abuf.assign(sizeof(uint16_t) * mfma_bf16_packed_elems(alt), 0);
            mfma_bf16_pack(alt, weight, reinterpret_cast<uint16_t*>(abuf.data()));
        }
    }
    bias.assign(pc.cout_pad, 0.f);
    for (int o = 0; o < cout; ++o) bias[o] = bias_in ? bias_in[o] : 0.f;
    hipError_t e = hipMalloc(&pc.w, wbytes);
    if (e == hipSuccess) e = hipMalloc((void**)&pc.b, sizeof(float) * bias.size());
    if (e == hipSuccess) e = hipMemcpy(pc.w, wbuf.data(), wbytes, hipMemcpyHostToDevice);
    if (e == hipSuccess && !abuf.empty()) {
        e = hipMalloc(&pc.w_alt, abuf.size());
        if (e == hipSuccess) e = hipMemcpy(pc.w_alt, abuf.data(), abuf.size(), hipMemcpyHostToDevice);
    }
    if (e == hipSuccess) e = hipMemcpy(pc.b, bias.data(), sizeof(float) * bias.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "uploading weights");
    return DSS_OK;
}

}  // namespace dss

using namespace dss;

// ------------------------------------------------------------------ misc

extern "C" const char* dss_status_string(dss_status s) {
    switch (s) {
        case DSS_OK: return "ok";
        case DSS_E_INVALID: return "invalid argument";
        case DSS_E_SHAPE: return "shape mismatch";
        case DSS_E_UNSUPPORTED: return "unsupported";
        case DSS_E_NOMEM: return "out of device memory";
        case DSS_E_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

extern "C" const char* dss_last_error(void) { return g_err.c_str(); }

extern "C" const char* dss_version(void) { return "0.1.0"; }

// ------------------------------------------------------------------ geometry

static void fill_geometry(const Chain& ch, const Geom& G, dss_dtype dt, dss_geometry* out) {
    std::memset(out, 0, sizeof *out);
    out->ndim = ch.ndim;
    out->in_c = ch.in_c;
    out->out_c = ch.out_c();
    out->n_chain = ch.L();
    out->B_h = ch.B_h;
    out->B_w = ch.B_w;
    out->K_h = ch.K_h();
    out->K_w = ch.K_w();
    out->r_h = G.r_h;
    out->r_w = G.r_w;
    out->D_h = G.D_h;
    out->D_w = G.D_w;
    out->out_h = G.out_h;
    out->out_w = G.out_w;
    out->dtype = dt;
    out->ell = G.ell;
    out->step_h = G.step_h;
    out->step_w = G.step_w;
    out->trim_h = G.trim_h;
    out->trim_w = G.trim_w;
    out->workspace_bytes = G.ws_bytes;
    out->conv_flops = G.conv_flops;
    out->pool_bytes = G.pool_bytes;
    out->total_bytes = G.total_bytes;
}

static dss_status fill_layer_geometry(const Chain& ch, const Geom& G, int j, dss_layer_geometry* out) {
    if (j < 0 || j > ch.L()) return fail(DSS_E_INVALID, "chain layer %d out of range 0..%d", j, ch.L());
    std::memset(out, 0, sizeof *out);
    out->kstar_h = ch.kstar_h[j];
    out->kstar_w = ch.kstar_w[j];
    out->u_h = ch.u_h[j];
    out->u_w = ch.u_w[j];
    if (j == 0) {
        out->c_h = out->c_w = out->k_h = out->k_w = 1;
        out->U_h = G.D_h;
        out->U_w = G.D_w;
        out->F = 1;
        out->channels = ch.in_c;
        return DSS_OK;
    }
    const ChainLayer& c = ch.layers[j - 1];
    const LayerGeom& lg = G.L[j - 1];
    out->c_h = c.c_h;
    out->c_w = c.c_w;
    out->k_h = c.k_h;
    out->k_w = c.k_w;
    out->U_h = lg.U_h;
    out->U_w = lg.U_w;
    out->F = lg.Fout_h * lg.Fout_w;
    out->channels = c.cout;
    out->has_conv = c.has_conv;
    out->has_pool = c.has_pool;
    out->relaxed = lg.relaxed;
    return DSS_OK;
}

extern "C" dss_status dss_chain_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                         int32_t in_channels, dss_dtype dtype, int32_t H, int32_t W,
                                         int32_t ell, dss_geometry* out) {
    if (!out) return fail(DSS_E_INVALID, "NULL output");
    if (dtype != DSS_F32 && dtype != DSS_BF16) return fail(DSS_E_UNSUPPORTED, "unknown dtype %d", dtype);
    Chain ch;
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &ch);
    if (s != DSS_OK) return s;
    Geom G;
    s = compute_geometry(ch, dtype, H, W, ell, &G);
    if (s != DSS_OK) return s;
    fill_geometry(ch, G, dtype, out);
    return DSS_OK;
}

extern "C" dss_status dss_chain_layer_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                               int32_t in_channels, int32_t H, int32_t W, int32_t ell, int32_t j,
                                               dss_layer_geometry* out) {
    if (!out) return fail(DSS_E_INVALID, "NULL output");
    Chain ch;
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &ch);
    if (s != DSS_OK) return s;
    Geom G;
    s = compute_geometry(ch, DSS_F32, H, W, ell, &G);
    if (s != DSS_OK) return s;
    return fill_layer_geometry(ch, G, j, out);
}

extern "C" dss_status dss_plan_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t ell, dss_geometry* out) {
    if (!plan || !out) return fail(DSS_E_INVALID, "NULL plan or output");
    Geom G;
    dss_status s = compute_geometry(plan->chain, plan->dtype, H, W, ell, &G);
    if (s != DSS_OK) return s;
    fill_geometry(plan->chain, G, plan->dtype, out);
    return DSS_OK;
}

extern "C" dss_status dss_plan_layer_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t ell, int32_t j,
                                              dss_layer_geometry* out) {
    if (!plan || !out) return fail(DSS_E_INVALID, "NULL plan or output");
    Geom G;
    dss_status s = compute_geometry(plan->chain, plan->dtype, H, W, ell, &G);
    if (s != DSS_OK) return s;
    return fill_layer_geometry(plan->chain, G, j, out);
}

// ------------------------------------------------------------------ plans

static void free_plan_memory(dss_plan* p) {
    for (auto* list : {&p->convs, &p->bconvs})
        for (auto& c : *list) {
            if (c.w) (void)hipFree(c.w);
            if (c.b) (void)hipFree(c.b);
            if (c.w_alt) (void)hipFree(c.w_alt);
            if (c.w2) (void)hipFree(c.w2);
            c.w = nullptr;
            c.b = nullptr;
            c.w_alt = nullptr;
            c.w2 = nullptr;
        }
    if (p->proj_b) (void)hipFree(p->proj_b);
    p->proj_b = nullptr;
    for (hipEvent_t e : p->events) (void)hipEventDestroy(e);
    p->events.clear();
    if (p->own_ws) (void)hipFree(p->own_ws);
    p->own_ws = nullptr;
    p->own_ws_bytes = 0;
}

extern "C" void dss_plan_destroy(dss_plan_t plan) {
    if (!plan) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    if (cur != plan->device) (void)hipSetDevice(plan->device);
    free_plan_memory(plan);
    if (cur != plan->device) (void)hipSetDevice(cur);
    delete plan;
}

// The fusions a plan uses (both can be turned off at plan creation, for
// cross-checks and A/B timing):
//  - the sliding max-pool + Frag of one-row fragments in the epilogue of the
//    convolution before it (decided per launch; DSS_FUSE_POOL=0 turns it off);
//  - the last chain layer, a 1x1 convolution to at most 4 channels with no
//    pool, folded into the epilogue of the convolution before it (an MFMA
//    convolution without a pool), with its weights uploaded in the layout that
//    epilogue reads (DSS_FUSE_PROJECTION=0 turns it off).
static dss_status setup_fusions(dss_plan* p, const dss_layer* layers) {
    const Chain& ch = p->chain;
    const int L = ch.L();
    const char* pool_env = getenv("DSS_FUSE_POOL");
    p->fuse_pool = !(pool_env && std::strcmp(pool_env, "0") == 0);
    const char* env = getenv("DSS_FUSE_PROJECTION");
    if (env && std::strcmp(env, "0") == 0) return DSS_OK;
    if (L < 2) return DSS_OK;
    const ChainLayer& a = ch.layers[L - 2];
    const ChainLayer& b = ch.layers[L - 1];
    if (!a.has_conv || a.has_pool || !b.has_conv || b.has_pool || b.c_h != 1 || b.c_w != 1 || b.cout > 4) return DSS_OK;
    PlanConv& pc = p->convs[L - 2];
    if (pc.impl != CONV_MFMA_F32 && pc.impl != CONV_MFMA_BF16) return DSS_OK;
    const int rows = std::max(pc.cout_pad, pc.cout_pad_alt);
    std::vector<float> w2((size_t)rows * 4, 0.f), b2(4, 0.f);
    const dss_layer& d = layers[b.desc];
    for (int n = 0; n < b.cin; ++n)
        for (int o = 0; o < b.cout; ++o) {
            float v = d.weight[(size_t)o * b.cin + n];
            if (p->dtype == DSS_BF16) {   // the plan's bfloat16 weights, as the unfused 1x1 convolution uses them
                const uint32_t u = (uint32_t)host_f32_to_bf16(v) << 16;
                std::memcpy(&v, &u, 4);
            }
            w2[(size_t)n * 4 + o] = v;
        }
    for (int o = 0; o < b.cout; ++o) b2[o] = d.bias ? d.bias[o] : 0.f;
    hipError_t e = hipMalloc((void**)&pc.w2, sizeof(float) * w2.size());
    if (e == hipSuccess) e = hipMalloc((void**)&p->proj_b, sizeof(float) * 4);
    if (e == hipSuccess) e = hipMemcpy(pc.w2, w2.data(), sizeof(float) * w2.size(), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemcpy(p->proj_b, b2.data(), sizeof(float) * 4, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "uploading the projection weights");
    p->fuse_proj = true;
    p->proj_cout = b.cout;
    p->proj_act = b.act;
    return DSS_OK;
}

extern "C" dss_status dss_plan_create(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                      int32_t in_channels, dss_dtype dtype, dss_plan_t* out_plan) {
    if (!out_plan) return fail(DSS_E_INVALID, "NULL out_plan");
    *out_plan = nullptr;
    if (dtype != DSS_F32 && dtype != DSS_BF16) return fail(DSS_E_UNSUPPORTED, "unknown dtype %d", dtype);
    dss_plan* p = new (std::nothrow) dss_plan;
    if (!p) return fail(DSS_E_NOMEM, "host allocation failed");
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &p->chain);
    if (s != DSS_OK) {
        delete p;
        return s;
    }
    p->dtype = dtype;
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) {
        delete p;
        return hip_fail(e, "hipGetDevice");
    }
    const int L = p->chain.L();
    p->convs.resize(L);
    if (dtype == DSS_F32) p->bconvs.resize(L);
    for (int j = 0; j < L; ++j) {
        const ChainLayer& c = p->chain.layers[j];
        if (!c.has_conv) continue;
        const dss_layer& d = layers[c.desc];
        s = upload_conv(c.cin, c.cout, c.c_h, c.c_w, c.act, d.weight, d.bias, dtype, p->convs[j]);
        if (s == DSS_OK && dtype == DSS_F32) {
            // input gradient: w'[i][o][t_h][t_w] = w[o][i][fh-1-t_h][fw-1-t_w]
            std::vector<float> wt((size_t)c.cin * c.cout * c.c_h * c.c_w);
            for (int o = 0; o < c.cout; ++o)
                for (int i = 0; i < c.cin; ++i)
                    for (int th = 0; th < c.c_h; ++th)
                        for (int tw = 0; tw < c.c_w; ++tw)
                            wt[(((size_t)i * c.cout + o) * c.c_h + (c.c_h - 1 - th)) * c.c_w + (c.c_w - 1 - tw)] =
                                d.weight[(((size_t)o * c.cin + i) * c.c_h + th) * c.c_w + tw];
            s = upload_conv(c.cout, c.cin, c.c_h, c.c_w, DSS_ACT_NONE, wt.data(), nullptr, dtype, p->bconvs[j]);
        }
        if (s != DSS_OK) {
            free_plan_memory(p);
            delete p;
            return s;
        }
    }
    s = setup_fusions(p, layers);
    if (s != DSS_OK) {
        free_plan_memory(p);
        delete p;
        return s;
    }
    *out_plan = p;
    return DSS_OK;
}

// ------------------------------------------------------------------ telemetry

extern "C" dss_status dss_plan_set_timing(dss_plan_t plan, int32_t enable) {
    if (!plan) return fail(DSS_E_INVALID, "NULL plan");
    if (!plan->recs.empty()) {
        // the events of earlier records may still be pending on some stream
        hipError_t e = hipEventSynchronize(plan->events[plan->recs.back().ev1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    }
    plan->timing = enable != 0;
    plan->recs.clear();
    return DSS_OK;
}

extern "C" dss_status dss_plan_timings(dss_plan_t plan, dss_launch_record* records, int32_t cap, int32_t* count) {
    if (!plan || !count || (cap > 0 && !records)) return fail(DSS_E_INVALID, "NULL argument");
    *count = (int32_t)plan->recs.size();
    for (int i = 0; i < (int)plan->recs.size() && i < cap; ++i) {
        const LaunchRec& r = plan->recs[i];
        hipError_t e = hipEventSynchronize(plan->events[r.ev1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, plan->events[r.ev0], plan->events[r.ev1]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        records[i].kernel = r.name;
        records[i].chain_layer = r.layer;
        records[i].tile_mode = r.tile_mode;
        records[i].ms = ms;
        records[i].flops = r.flops;
        records[i].bytes = r.bytes;
    }
    return DSS_OK;
}

namespace {

// Brackets each launch with HIP events when the plan's timing is on.
struct Timer {
    dss_plan* p;
    hipStream_t s;
    int next = 0;
    bool on;
    // timed: false for evaluations that must not create events (allocation-free entry points)
    Timer(dss_plan* p_, hipStream_t s_, bool timed = true) : p(p_), s(s_), on(timed && p_->timing) {
        next = 2 * (int)p->recs.size();
    }
    hipError_t event(int* idx) {
        if (next >= (int)p->events.size()) {
            hipEvent_t ev;
            hipError_t e = hipEventCreate(&ev);
            if (e != hipSuccess) return e;
            p->events.push_back(ev);
        }
        *idx = next++;
        return hipEventRecord(p->events[*idx], s);
    }
    template <class F>
    hipError_t run(const char* name, int layer, double flops, double bytes, F&& launch, int tile_mode = -1) {
        if (!on) return launch();
        LaunchRec r{name, layer, flops, bytes, 0, 0, tile_mode};
        hipError_t e = event(&r.ev0);
        if (e != hipSuccess) return e;
        e = launch();
        if (e != hipSuccess) return e;
        e = event(&r.ev1);
        if (e != hipSuccess) return e;
        p->recs.push_back(r);
        return hipSuccess;
    }
};

// Telemetry name of a convolution launch: one name per kernel instantiation, so
// that per-name averages match a profiler's per-symbol statistics.
const char* conv_name(const PlanConv& pc, dss_dtype tout) {
    switch (pc.impl) {
        case CONV_MFMA_F32:
            return pc.bn == 128 ? "conv_mfma_f32_n128" : pc.bn == 64 ? "conv_mfma_f32_n64" : "conv_mfma_f32_n32";
        case CONV_MFMA_BF16:
            if (tout == DSS_F32)
                return pc.bn == 128 ? "conv_mfma_bf16_n128_f32out" : pc.bn == 64 ? "conv_mfma_bf16_n64_f32out"
                                                                   : "conv_mfma_bf16_n32_f32out";
            return pc.bn == 128 ? "conv_mfma_bf16_n128" : pc.bn == 64 ? "conv_mfma_bf16_n64" : "conv_mfma_bf16_n32";
        default:
            // the direct kernel's forms for few outputs and many inputs: lanes over
            // input channels, or LDS-staged tiles
            if (conv_lanesum_ok(pc.cin, pc)) return "conv_lanesum";
            return pc.cin >= 16 && pc.cout_pad <= 8 ? "conv_narrow" : "conv_direct";
    }
}

// Telemetry name of a convolution launch with the folded projection.
const char* conv_proj_name(const PlanConv& pc) {
    if (pc.impl == CONV_MFMA_F32)
        return pc.bn == 128 ? "conv_mfma_f32_n128_proj" : pc.bn == 64 ? "conv_mfma_f32_n64_proj"
                                                                      : "conv_mfma_f32_n32_proj";
    return pc.bn == 128 ? "conv_mfma_bf16_n128_proj" : pc.bn == 64 ? "conv_mfma_bf16_n64_proj"
                                                                   : "conv_mfma_bf16_n32_proj";
}

}  // namespace

// Runs Stuff and chain layers 1..upto.  On return *cur points at the last
// tensor (channels-last fragment layout) and *cur_dt is its element type.
// Chain layers 1..upto on the packed input in buf[0] (the two halves of the
// workspace ping-pong).  On return *cur points at the last tensor (channels-last
// fragment layout) and *cur_dt is its element type.  A relaxed layer's pooling
// runs over all Fin fragments at once as one tall signal of Fin * E_h rows:
// every fragment's extent is a multiple of k_h, so no block straddles two.
// With fold (and a plan that folds its projection, upto = L), the convolution of
// layer L - 1 writes the partial projections instead of its activations, layer
// L is skipped, and *part_nbs receives the number of channel groups summed
// later (0 when nothing was folded).
static dss_status run_layers(dss_plan* p, const Geom& G, int upto, char* const buf[2], hipStream_t stream, Timer& T,
                             void** cur_out, dss_dtype* cur_dt, bool fold = false, int* part_nbs = nullptr) {
    const Chain& ch = p->chain;
    int which = 0;
    const dss_dtype dt = p->dtype;
    const double es = (double)dtype_size(dt);
    hipError_t e;
    void* cur = buf[0];
    dss_dtype cdt = dt;
    if (part_nbs) *part_nbs = 0;
    const bool folding = fold && p->fuse_proj && upto == ch.L() && part_nbs;
    for (int j = 1; j <= upto; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        const LayerGeom& lg = G.L[j - 1];
        const int Fin = lg.Fin_h * lg.Fin_w;
        const PlanConv fpc = folding && j == ch.L() - 1
                                 ? mfma_launch_variant(p->convs[j - 1], Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w)
                                 : PlanConv{};
        // the partial projections (16 bytes per sample and channel group of 64,
        // or 32 for the 32-channel N tile) must fit a ping-pong half, which
        // holds at least this layer's output
        const int ngroups = fpc.w2 ? fpc.cout_pad / (fpc.bn == 32 ? 32 : 64) : 0;
        if (fpc.w2 && (int64_t)ngroups * Fin * lg.E_h * lg.E_w * 16 <= G.buf_bytes) {
            // conv T_{L-1} with the 1x1 projection T_L folded into its epilogue
            const PlanConv& pc = fpc;
            const ChainLayer& cl = ch.layers[j];
            void* dst = buf[which ^ 1];
            const double f1 = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const double f2 = 2.0 * Fin * (double)lg.E_h * lg.E_w * cl.cout * (double)cl.cin;
            const int nbs = ngroups;
            const double bytes = (double)Fin * lg.Uin_h * lg.Uin_w * c.cin * dtype_size(cdt) +
                                 (double)nbs * Fin * lg.E_h * lg.E_w * 16.0 +
                                 (double)c.cout * c.cin * c.c_h * c.c_w * es;
            e = T.run(
                conv_proj_name(pc), j, f1 + f2, bytes,
                [&] {
                    return launch_conv_mfma_proj(cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w, pc, (float*)dst,
                                                 stream);
                },
                T.on ? mfma_tile_mode(pc, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w) : -1);
            if (e != hipSuccess) return hip_fail(e, "conv + projection launch");
            *part_nbs = nbs;
            *cur_out = dst;
            *cur_dt = DSS_F32;
            return DSS_OK;
        }
        if (c.has_conv && c.has_pool && p->fuse_pool && !lg.relaxed && !lg.dilated && lg.E_h == 1 && lg.Fin_h == 1 &&
            c.k_h == 1 && c.k_w >= 2 && c.k_w <= 4 && p->convs[j - 1].impl == CONV_DIRECT && c.c_h == 1 && c.cin < 16) {
            // one-row fragments with few input channels (the first layer of a 1-D
            // chain; every fashion runs such a layer on the plain direct kernel,
            // whose summation order the fused kernel keeps): each thread computes
            // k outputs and writes their maximum straight to its fragment
            const PlanConv& pc = p->convs[j - 1];
            void* dst = buf[which ^ 1];
            const double flops = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const double bytes = (double)Fin * lg.Uin_h * lg.Uin_w * c.cin * dtype_size(cdt) +
                                 (double)lg.Fout_h * lg.Fout_w * lg.U_h * lg.U_w * c.cout * dtype_size(cdt) +
                                 (double)c.cout * c.cin * c.c_h * c.c_w * es;
            e = T.run("conv_direct_pool", j, flops, bytes, [&] {
                return launch_conv_direct_pool(cdt, cur, Fin, lg.Uin_w, c.cin, pc, c.k_w, lg.U_w, dst, stream);
            });
            if (e != hipSuccess) return hip_fail(e, "conv + pool launch");
            which ^= 1;
            cur = dst;
            continue;
        }
        if (c.has_conv && c.has_pool && p->fuse_pool && !lg.relaxed && !lg.dilated && lg.E_h == 1 && lg.Fin_h == 1 &&
            c.k_h == 1 && c.k_w >= 2 && c.cout % 4 == 0) {
            // one-row fragments: the sliding max-pool and Frag in the convolution's
            // epilogue, on spatial tiles of 256 samples stepped by 257 - k; taken
            // when those tiles compute at most 10 % more samples than the layer has
            const PlanConv pc = mfma_launch_variant(p->convs[j - 1], Fin, lg.Uin_h, lg.Uin_w, 1, 1);
            const int64_t tiles = ((int64_t)c.k_w * lg.U_w + 256 - c.k_w) / (256 - c.k_w + 1);
            if (pc.impl == CONV_MFMA_F32 && pc.bn <= 64 && 10 * tiles * 256 <= 11 * (int64_t)lg.E_w) {
                void* dst = buf[which ^ 1];
                const double flops = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
                const double bytes = (double)Fin * lg.Uin_h * lg.Uin_w * c.cin * 4.0 +
                                     (double)lg.Fout_h * lg.Fout_w * lg.U_h * lg.U_w * c.cout * 4.0 +
                                     (double)c.cout * c.cin * c.c_h * c.c_w * 4.0;
                e = T.run(pc.bn == 64 ? "conv_mfma_f32_n64_pool" : "conv_mfma_f32_n32_pool", j, flops, bytes,
                          [&] {
                              return launch_conv_mfma_pool((const float*)cur, Fin, lg.Uin_h, lg.Uin_w, pc, c.k_w,
                                                           (float*)dst, stream);
                          },
                          T.on ? 0 : -1);
                if (e != hipSuccess) return hip_fail(e, "conv + pool launch");
                which ^= 1;
                cur = dst;
                continue;
            }
        }
        if (c.has_conv) {
            const PlanConv pc = mfma_launch_variant(p->convs[j - 1], Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w);
            const bool last_op = (j == ch.L()) && !c.has_pool;
            const dss_dtype tout = (dt == DSS_BF16 && last_op) ? DSS_F32 : dt;
            void* dst = buf[which ^ 1];
            const double flops = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const double bytes = (double)Fin * lg.Uin_h * lg.Uin_w * c.cin * dtype_size(cdt) +
                                 (double)Fin * lg.E_h * lg.E_w * c.cout * dtype_size(tout) +
                                 (double)c.cout * c.cin * c.c_h * c.c_w * es;
            e = T.run(
                conv_name(pc, tout), j, flops, bytes,
                [&]() -> hipError_t {
                    if (pc.impl == CONV_MFMA_F32)
                        return launch_conv_mfma_f32((const float*)cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w,
                                                    pc, (float*)dst, stream);
                    if (pc.impl == CONV_MFMA_BF16)
                        return launch_conv_mfma_bf16(tout, (const uint16_t*)cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h,
                                                     lg.dil_w, pc, dst, stream);
                    return launch_conv_direct(cdt, tout, cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w, c.cin, pc,
                                              dst, stream);
                },
                T.on ? mfma_tile_mode(pc, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w) : -1);
            if (e != hipSuccess) return hip_fail(e, "conv launch");
            which ^= 1;
            cur = dst;
            cdt = tout;
        }
        if (c.has_pool && lg.dilated) {
            void* dst = buf[which ^ 1];
            const double bytes = ((double)lg.E_h * lg.E_w + (double)lg.U_h * lg.U_w) * c.cout * dtype_size(cdt);
            e = T.run("pool_dilate", j, 0.0, bytes, [&] {
                return launch_pool_dilate(cdt, cur, lg.E_h, lg.E_w, c.cout, c.k_h, c.k_w, lg.dil_h, lg.dil_w, dst,
                                          stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pool_dilate launch");
            which ^= 1;
            cur = dst;
        } else if (c.has_pool && lg.relaxed) {
            void* dst = buf[which ^ 1];
            const double bytes = (double)Fin * ((double)lg.E_h * lg.E_w + (double)lg.U_h * lg.U_w) * c.cout *
                                 dtype_size(cdt);
            e = T.run("pool_stride", j, 0.0, bytes, [&] {
                return launch_pool_stride(cdt, cur, Fin * lg.E_h, lg.E_w, c.cout, c.k_h, c.k_w, dst, stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pool_stride launch");
            which ^= 1;
            cur = dst;
        } else if (c.has_pool) {
            void* dst = buf[which ^ 1];
            const double bytes = ((double)Fin * lg.E_h * lg.E_w + (double)lg.Fout_h * lg.Fout_w * lg.U_h * lg.U_w) *
                                 c.cout * dtype_size(cdt);
            e = T.run("pool_frag", j, 0.0, bytes, [&] {
                return launch_pool_frag(cdt, cur, lg.Fin_h, lg.Fin_w, lg.E_h, lg.E_w, c.cout, c.k_h, c.k_w, dst, stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pool_frag launch");
            which ^= 1;
            cur = dst;
        }
    }
    *cur_out = cur;
    *cur_dt = cdt;
    return DSS_OK;
}

// Stuff (or trim) into the workspace, then chain layers 1..upto.
static dss_status run_chain(dss_plan* p, const Geom& G, const void* signal, int upto, char* ws,
                            hipStream_t stream, Timer& T, void** cur_out, dss_dtype* cur_dt, bool fold = false,
                            int* part_nbs = nullptr) {
    const Chain& ch = p->chain;
    char* const buf[2] = {ws, ws + G.buf_bytes};
    const dss_dtype dt = p->dtype;
    const double es = (double)dtype_size(dt);
    const double in_read = (double)std::min(G.H, G.D_h) * std::min(G.W, G.D_w);
    hipError_t e = T.run("stuff_pack", 0, 0.0, (double)ch.in_c * (in_read + G.D_h * (double)G.D_w) * es,
                         [&] { return launch_stuff_pack(dt, signal, ch.in_c, G.H, G.W, buf[0], G.D_h, G.D_w, stream); });
    if (e != hipSuccess) return hip_fail(e, "stuff_pack launch");
    return run_layers(p, G, upto, buf, stream, T, cur_out, cur_dt, fold, part_nbs);
}

// Checks that the plan belongs to the current device.
static dss_status check_device(const dss_plan* plan) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != plan->device)
        return fail(DSS_E_INVALID, "plan belongs to device %d but device %d is current", plan->device, cur);
    return DSS_OK;
}

// The workspace an evaluation runs in: the caller's (at least `need` bytes,
// 256-byte aligned), or, for workspace == NULL, the plan's own buffer, grown to
// `need` bytes if it is smaller.  Growing first waits for the device, since work
// enqueued earlier may still use the old buffer.  Called after every other
// argument check, so a failure here (DSS_E_NOMEM, DSS_E_HIP) still leaves
// nothing enqueued.
static dss_status resolve_workspace(dss_plan* plan, void* workspace, int64_t workspace_bytes, int64_t need,
                                    char** ws) {
    if (workspace) {
        if (workspace_bytes < need)
            return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                        (long long)workspace_bytes, (long long)need);
        if (((uintptr_t)workspace & 255u) != 0) return fail(DSS_E_INVALID, "workspace is not 256-byte aligned");
        *ws = (char*)workspace;
        return DSS_OK;
    }
    std::lock_guard<std::mutex> lock(plan->ws_mu);
    if (plan->own_ws_bytes < need) {
        if (plan->own_ws) {
            hipError_t e = hipDeviceSynchronize();
            if (e != hipSuccess) return hip_fail(e, "waiting for the device before growing the plan's workspace");
            e = hipFree(plan->own_ws);
            plan->own_ws = nullptr;
            plan->own_ws_bytes = 0;
            if (e != hipSuccess) return hip_fail(e, "freeing the plan's workspace");
        }
        const int64_t bytes = std::max<int64_t>(need, 256);
        hipError_t e = hipMalloc(&plan->own_ws, (size_t)bytes);
        if (e != hipSuccess) {
            plan->own_ws = nullptr;
            return hip_fail(e, "allocating the plan's workspace");
        }
        plan->own_ws_bytes = bytes;
    }
    *ws = (char*)plan->own_ws;
    return DSS_OK;
}

static dss_status check_eval_args(dss_plan_t plan, const void* signal, const void* out, void* workspace,
                                  int64_t workspace_bytes, int32_t H, int32_t W, int32_t ell, Geom* G, char** ws) {
    dss_status s = dss::eval_prepare(plan, signal, out, H, W, ell, G);
    if (s != DSS_OK) return s;
    if (workspace && workspace_bytes < G->ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G->ws_bytes);
    return resolve_workspace(plan, workspace, workspace_bytes, G->ws_bytes, ws);
}

namespace dss {

dss_status eval_prepare(dss_plan_t plan, const void* signal, const void* out, int H, int W, int ell, Geom* G) {
    if (!plan || !signal || !out) return fail(DSS_E_INVALID, "NULL plan, signal or out");
    dss_status s = compute_geometry(plan->chain, plan->dtype, H, W, ell, G);
    if (s != DSS_OK) return s;
    return check_device(plan);
}

dss_status eval_run(dss_plan_t plan, const Geom& G, const void* signal, float* out, char* ws, hipStream_t stream,
                    bool timed) {
    Timer T(plan, stream, timed);
    void* cur = nullptr;
    dss_dtype cdt;
    int part_nbs = 0;
    dss_status s = run_chain(plan, G, signal, plan->chain.L(), ws, stream, T, &cur, &cdt, true, &part_nbs);
    if (s != DSS_OK) return s;
    const Chain& ch = plan->chain;
    // Defrag_{k*_L / k*_ell}, then keep the first out_h x out_w samples (this is
    // Trim_r of the dense evaluation and the final trimming of the stuffing mode)
    const int Gh = ch.K_h() / G.step_h, Gw = ch.K_w() / G.step_w;
    const int Uh = G.L.back().U_h, Uw = G.L.back().U_w;
    if (part_nbs > 0) {
        // the folded projection: sum the channel groups' partial dot products, + bias, activation
        const double bytes = (double)part_nbs * Gh * Gw * Uh * Uw * 16.0 + (double)G.out_h * G.out_w * ch.out_c() * 4.0;
        hipError_t e = T.run("defrag_sum", ch.L() + 1, 0.0, bytes, [&] {
            return launch_defrag_sum((const float*)cur, part_nbs, Gh, Gw, Uh, Uw, ch.out_c(), plan->proj_b,
                                     plan->proj_act, out, G.out_h, G.out_w, stream);
        });
        if (e != hipSuccess) return hip_fail(e, "defrag_sum launch");
        return DSS_OK;
    }
    const double bytes = (double)Gh * Gw * Uh * Uw * ch.out_c() * dtype_size(cdt) +
                         (double)G.out_h * G.out_w * ch.out_c() * 4.0;
    hipError_t e = T.run("defrag_trim", ch.L() + 1, 0.0, bytes, [&] {
        return launch_defrag_trim(cdt, cur, Gh, Gw, Uh, Uw, ch.out_c(), out, G.out_h, G.out_w, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "defrag_trim launch");
    return DSS_OK;
}

}  // namespace dss

extern "C" dss_status dss_eval_mixed(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                                     float* out, void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    Geom G;
    char* ws = nullptr;
    dss_status s = check_eval_args(plan, signal, out, workspace, workspace_bytes, H, W, ell, &G, &ws);
    if (s != DSS_OK) return s;
    return eval_run(plan, G, signal, out, ws, stream, true);
}

extern "C" dss_status dss_eval_dense(dss_plan_t plan, const void* signal, int32_t H, int32_t W, float* out,
                                     void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    return dss_eval_mixed(plan, signal, H, W, 0, out, workspace, workspace_bytes, stream);
}

extern "C" dss_status dss_eval_slide(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                                     int32_t j, float* out, void* workspace, int64_t workspace_bytes,
                                     hipStream_t stream) {
    if (plan && (j < 0 || j > plan->chain.L()))
        return fail(DSS_E_INVALID, "chain layer %d out of range 0..%d", j, plan->chain.L());
    Geom G;
    char* ws = nullptr;
    dss_status s = check_eval_args(plan, signal, out, workspace, workspace_bytes, H, W, ell, &G, &ws);
    if (s != DSS_OK) return s;
    Timer T(plan, stream);
    void* cur = nullptr;
    dss_dtype cdt;
    s = run_chain(plan, G, signal, j, ws, stream, T, &cur, &cdt);
    if (s != DSS_OK) return s;
    const Chain& ch = plan->chain;
    const int F = j == 0 ? 1 : G.L[j - 1].Fout_h * G.L[j - 1].Fout_w;
    const int h = j == 0 ? G.D_h : G.L[j - 1].U_h;
    const int w = j == 0 ? G.D_w : G.L[j - 1].U_w;
    const int C = j == 0 ? ch.in_c : ch.layers[j - 1].cout;
    hipError_t e = T.run("to_planar", j, 0.0, 0.0, [&] { return launch_to_planar(cdt, cur, F, h, w, C, out, stream); });
    if (e != hipSuccess) return hip_fail(e, "to_planar launch");
    return DSS_OK;
}

// ------------------------------------------------------------------ EvalStride baseline

extern "C" dss_status dss_chain_stride_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                                int32_t in_channels, dss_dtype dtype, int32_t count,
                                                int64_t* workspace_bytes, double* conv_flops) {
    if (!workspace_bytes) return fail(DSS_E_INVALID, "NULL output");
    if (dtype != DSS_F32 && dtype != DSS_BF16) return fail(DSS_E_UNSUPPORTED, "unknown dtype %d", dtype);
    Chain ch;
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &ch);
    if (s != DSS_OK) return s;
    Geom G;
    s = compute_stride_geometry(ch, dtype, count, &G);
    if (s != DSS_OK) return s;
    *workspace_bytes = G.ws_bytes;
    if (conv_flops) *conv_flops = G.conv_flops;
    return DSS_OK;
}

extern "C" dss_status dss_plan_stride_geometry(dss_plan_t plan, int32_t count, int64_t* workspace_bytes,
                                               double* conv_flops) {
    if (!plan || !workspace_bytes) return fail(DSS_E_INVALID, "NULL plan or output");
    Geom G;
    dss_status s = compute_stride_geometry(plan->chain, plan->dtype, count, &G);
    if (s != DSS_OK) return s;
    *workspace_bytes = G.ws_bytes;
    if (conv_flops) *conv_flops = G.conv_flops;
    return DSS_OK;
}

extern "C" dss_status dss_eval_stride(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int64_t first,
                                      int32_t count, float* out, void* workspace, int64_t workspace_bytes,
                                      hipStream_t stream) {
    if (!plan || !signal || !out) return fail(DSS_E_INVALID, "NULL plan, signal or out");
    const Chain& ch = plan->chain;
    if (ch.ndim == 1 && H != 1) return fail(DSS_E_SHAPE, "1-D plan needs H = 1 (got %d)", H);
    if (H < ch.B_h || W < ch.B_w)
        return fail(DSS_E_SHAPE, "signal %dx%d is smaller than the receptive field %dx%d", H, W, ch.B_h, ch.B_w);
    const int O_h = H - ch.B_h + 1, O_w = W - ch.B_w + 1;
    if (first < 0 || count <= 0 || first + count > (int64_t)O_h * O_w)
        return fail(DSS_E_INVALID, "windows [%lld, %lld) outside 0..%lld", (long long)first,
                    (long long)(first + count), (long long)O_h * O_w);
    Geom G;
    dss_status s = compute_stride_geometry(ch, plan->dtype, count, &G);
    if (s != DSS_OK) return s;
    if (workspace && workspace_bytes < G.ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G.ws_bytes);
    s = check_device(plan);
    if (s != DSS_OK) return s;
    char* ws = nullptr;
    s = resolve_workspace(plan, workspace, workspace_bytes, G.ws_bytes, &ws);
    if (s != DSS_OK) return s;
    hipError_t e;

    Timer T(plan, stream);
    char* const buf[2] = {ws, ws + G.buf_bytes};
    const double es = (double)dtype_size(plan->dtype);
    const double pbytes = 2.0 * count * (double)ch.B_h * ch.B_w * ch.in_c * es;
    e = T.run("patch_pack", 0, 0.0, pbytes, [&] {
        return launch_patch_pack(plan->dtype, signal, ch.in_c, H, W, O_w, first, count, ch.B_h, ch.B_w, buf[0],
                                 stream);
    });
    if (e != hipSuccess) return hip_fail(e, "patch_pack launch");
    void* cur = nullptr;
    dss_dtype cdt;
    int part_nbs = 0;
    s = run_layers(plan, G, ch.L(), buf, stream, T, &cur, &cdt, true, &part_nbs);
    if (s != DSS_OK) return s;
    if (part_nbs > 0) {
        const double pbytes = (double)count * (part_nbs * 16.0 + ch.out_c() * 4.0);
        e = T.run("window_scatter_sum", ch.L() + 1, 0.0, pbytes, [&] {
            return launch_window_scatter_sum((const float*)cur, part_nbs, count, ch.out_c(), plan->proj_b,
                                             plan->proj_act, first, (int64_t)O_h * O_w, out, stream);
        });
        if (e != hipSuccess) return hip_fail(e, "window_scatter_sum launch");
        return DSS_OK;
    }
    const double sbytes = (double)count * ch.out_c() * (dtype_size(cdt) + 4.0);
    e = T.run("window_scatter", ch.L() + 1, 0.0, sbytes, [&] {
        return launch_window_scatter(cdt, cur, count, ch.out_c(), first, (int64_t)O_h * O_w, out, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "window_scatter launch");
    return DSS_OK;
}

// ------------------------------------------------------------------ dilated fashion

static dss_status dilate_geometry_out(const Chain& ch, const Geom& G, int j, int32_t* V_h, int32_t* V_w,
                                      int64_t* workspace_bytes, double* conv_flops) {
    if (j < 0 || j > ch.L()) return fail(DSS_E_INVALID, "chain layer %d out of range 0..%d", j, ch.L());
    if (V_h) *V_h = j == 0 ? G.H : G.L[j - 1].U_h;
    if (V_w) *V_w = j == 0 ? G.W : G.L[j - 1].U_w;
    if (workspace_bytes) *workspace_bytes = G.ws_bytes;
    if (conv_flops) *conv_flops = G.conv_flops;
    return DSS_OK;
}

extern "C" dss_status dss_chain_dilate_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                                int32_t in_channels, dss_dtype dtype, int32_t H, int32_t W, int32_t j,
                                                int32_t* V_h, int32_t* V_w, int64_t* workspace_bytes,
                                                double* conv_flops) {
    if (dtype != DSS_F32 && dtype != DSS_BF16) return fail(DSS_E_UNSUPPORTED, "unknown dtype %d", dtype);
    Chain ch;
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &ch);
    if (s != DSS_OK) return s;
    Geom G;
    s = compute_dilate_geometry(ch, dtype, H, W, &G);
    if (s != DSS_OK) return s;
    return dilate_geometry_out(ch, G, j, V_h, V_w, workspace_bytes, conv_flops);
}

extern "C" dss_status dss_plan_dilate_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t j, int32_t* V_h,
                                               int32_t* V_w, int64_t* workspace_bytes, double* conv_flops) {
    if (!plan) return fail(DSS_E_INVALID, "NULL plan");
    Geom G;
    dss_status s = compute_dilate_geometry(plan->chain, plan->dtype, H, W, &G);
    if (s != DSS_OK) return s;
    return dilate_geometry_out(plan->chain, G, j, V_h, V_w, workspace_bytes, conv_flops);
}

extern "C" dss_status dss_eval_dilate(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t j, float* out,
                                      void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    if (!plan || !signal || !out) return fail(DSS_E_INVALID, "NULL plan, signal or out");
    const Chain& ch = plan->chain;
    if (j < 0 || j > ch.L()) return fail(DSS_E_INVALID, "chain layer %d out of range 0..%d", j, ch.L());
    Geom G;
    dss_status s = compute_dilate_geometry(ch, plan->dtype, H, W, &G);
    if (s != DSS_OK) return s;
    if (workspace && workspace_bytes < G.ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G.ws_bytes);
    s = check_device(plan);
    if (s != DSS_OK) return s;
    char* ws = nullptr;
    s = resolve_workspace(plan, workspace, workspace_bytes, G.ws_bytes, &ws);
    if (s != DSS_OK) return s;
    hipError_t e;
    Timer T(plan, stream);
    void* cur = nullptr;
    dss_dtype cdt;
    int part_nbs = 0;
    s = run_chain(plan, G, signal, j, ws, stream, T, &cur, &cdt, true, &part_nbs);   // D = H x W: a plain pack
    if (s != DSS_OK) return s;
    const int h = j == 0 ? H : G.L[j - 1].U_h;
    const int w = j == 0 ? W : G.L[j - 1].U_w;
    const int C = j == 0 ? ch.in_c : ch.layers[j - 1].cout;
    if (part_nbs > 0) {
        const double pbytes = (double)h * w * (part_nbs * 16.0 + C * 4.0);
        e = T.run("planar_sum", ch.L() + 1, 0.0, pbytes, [&] {
            return launch_planar_sum((const float*)cur, part_nbs, h, w, C, plan->proj_b, plan->proj_act, out, stream);
        });
        if (e != hipSuccess) return hip_fail(e, "planar_sum launch");
        return DSS_OK;
    }
    const double bytes = (double)h * w * C * (dtype_size(cdt) + 4.0);
    e = T.run("to_planar", ch.L() + 1, 0.0, bytes, [&] { return launch_to_planar(cdt, cur, 1, h, w, C, out, stream); });
    if (e != hipSuccess) return hip_fail(e, "to_planar launch");
    return DSS_OK;
}

// ------------------------------------------------------------------ backward

namespace {

// Workspace layout and work of the backward pass for one signal extent.
struct BwdLayout {
    Geom G;                                  // dense geometry (ell = 0)
    std::vector<int64_t> a_off, c_off;       // byte offsets: A_0..A_L, conv outputs C_1..C_L
    int64_t g_off[2] = {0, 0}, pad_off = 0, wpart_off = 0, total = 0;
    std::vector<WgradPlan> wg;               // per chain layer with a convolution
    std::vector<int64_t> wofs, bofs;         // float offsets of each conv's gradients in the outputs
    int64_t wfloats = 0, bfloats = 0;
    double flops = 0;                        // forward + weight-gradient + input-gradient convolutions
};

int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

// plan: the plan whose input-gradient convolutions run (their kernels decide
// whether a zero-bordered copy of the gradient is needed), or NULL for a chain
// alone (the kernels the chain's plan would choose).
dss_status backward_layout(const Chain& ch, int H, int W, bool want_dx, BwdLayout* out,
                           const dss_plan* plan = nullptr) {
    BwdLayout B;
    dss_status s = compute_geometry(ch, DSS_F32, H, W, 0, &B.G);
    if (s != DSS_OK) return s;
    const Geom& G = B.G;
    const int L = ch.L();
    int64_t off = 0;
    auto take = [&](int64_t bytes) { const int64_t o = off; off += align256(bytes); return o; };
    std::vector<int64_t> asz(L + 1), csz(L + 1, 0);
    asz[0] = (int64_t)G.D_h * G.D_w * ch.in_c * 4;
    B.a_off.assign(L + 1, 0);
    B.c_off.assign(L + 1, 0);
    B.a_off[0] = take(asz[0]);
    int64_t gmax = asz[0], padmax = 0, wpmax = 0;
    B.wg.resize(L + 1);
    B.wofs.assign(L + 1, -1);
    B.bofs.assign(L + 1, -1);
    for (int j = 1; j <= L; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        const LayerGeom& lg = G.L[j - 1];
        const int64_t Fin = (int64_t)lg.Fin_h * lg.Fin_w, Fout = (int64_t)lg.Fout_h * lg.Fout_w;
        if (c.has_conv) csz[j] = Fin * lg.E_h * lg.E_w * c.cout * 4;
        asz[j] = c.has_pool ? Fout * lg.U_h * lg.U_w * c.cout * 4 : csz[j];
        if (c.has_conv && c.has_pool) B.c_off[j] = take(csz[j]);
        B.a_off[j] = take(asz[j]);
        if (c.has_conv && !c.has_pool) B.c_off[j] = B.a_off[j];
        if (!c.has_conv) B.c_off[j] = B.a_off[j - 1];
        gmax = std::max({gmax, asz[j], csz[j], asz[j - 1]});
        if (c.has_conv) {
            const double f = 2.0 * Fin * lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            B.flops += 2.0 * f;                           // forward + weight gradient
            if (j > 1 || want_dx) {
                B.flops += f;                             // input gradient
                // the MFMA kernel reads the gradient with a virtual zero border;
                // the direct kernel needs it written out
                const ConvImpl bi = plan && (int)plan->bconvs.size() >= j ? plan->bconvs[j - 1].impl
                                                                           : choose_impl(c.cout, c.cin, c.c_h, c.c_w,
                                                                                         DSS_F32);
                if (bi == CONV_DIRECT)
                    padmax = std::max(padmax, Fin * (lg.E_h + 2 * (c.c_h - 1)) *
                                                  (int64_t)(lg.E_w + 2 * (c.c_w - 1)) * c.cout * 4);
            }
            B.wg[j] = wgrad_plan((int)Fin, lg.E_h, lg.E_w, c.cout, c.cin, c.c_h, c.c_w);
            wpmax = std::max(wpmax, (B.wg[j].partial_floats + B.wg[j].bias_partial_floats) * 4);
            B.wofs[j] = B.wfloats;
            B.bofs[j] = B.bfloats;
            B.wfloats += (int64_t)c.cout * c.cin * c.c_h * c.c_w;
            B.bfloats += c.cout;
        }
    }
    B.g_off[0] = take(gmax);
    B.g_off[1] = take(gmax);
    B.pad_off = take(std::max<int64_t>(padmax, 256));
    B.wpart_off = take(std::max<int64_t>(wpmax, 256));
    B.total = off;
    *out = std::move(B);
    return DSS_OK;
}

const char* dgrad_name(const PlanConv& pc) {
    switch (pc.impl) {
        case CONV_MFMA_F32:
            return pc.bn == 128 ? "dgrad_mfma_f32_n128" : pc.bn == 64 ? "dgrad_mfma_f32_n64" : "dgrad_mfma_f32_n32";
        default:
            return "dgrad_direct";
    }
}

}  // namespace

static dss_status backward_geometry_out(const BwdLayout& B, int64_t* ws, int64_t* wf, int64_t* bf, double* flops) {
    if (ws) *ws = B.total;
    if (wf) *wf = B.wfloats;
    if (bf) *bf = B.bfloats;
    if (flops) *flops = B.flops;
    return DSS_OK;
}

extern "C" dss_status dss_chain_backward_geometry(const dss_layer* layers, int32_t n_layers, int32_t ndim,
                                                  int32_t in_channels, int32_t H, int32_t W, int32_t with_signal_grad,
                                                  int64_t* workspace_bytes, int64_t* weight_grad_floats,
                                                  int64_t* bias_grad_floats, double* flops) {
    Chain ch;
    dss_status s = build_chain(layers, n_layers, ndim, in_channels, &ch);
    if (s != DSS_OK) return s;
    BwdLayout B;
    s = backward_layout(ch, H, W, with_signal_grad != 0, &B);
    if (s != DSS_OK) return s;
    return backward_geometry_out(B, workspace_bytes, weight_grad_floats, bias_grad_floats, flops);
}

extern "C" dss_status dss_plan_backward_geometry(dss_plan_t plan, int32_t H, int32_t W, int32_t with_signal_grad,
                                                 int64_t* workspace_bytes, int64_t* weight_grad_floats,
                                                 int64_t* bias_grad_floats, double* flops) {
    if (!plan) return fail(DSS_E_INVALID, "NULL plan");
    BwdLayout B;
    dss_status s = backward_layout(plan->chain, H, W, with_signal_grad != 0, &B, plan);
    if (s != DSS_OK) return s;
    return backward_geometry_out(B, workspace_bytes, weight_grad_floats, bias_grad_floats, flops);
}

extern "C" dss_status dss_backward_dense(dss_plan_t plan, const void* signal, int32_t H, int32_t W,
                                         const float* grad_out, float* grad_weight, float* grad_bias,
                                         float* grad_signal, void* workspace, int64_t workspace_bytes,
                                         hipStream_t stream) {
    if (!plan || !signal || !grad_out || !grad_weight || !grad_bias)
        return fail(DSS_E_INVALID, "NULL plan, signal, grad_out, grad_weight or grad_bias");
    if (plan->dtype != DSS_F32) return fail(DSS_E_UNSUPPORTED, "the backward pass is implemented for binary32 plans");
    const Chain& ch = plan->chain;
    BwdLayout B;
    dss_status s = backward_layout(ch, H, W, grad_signal != nullptr, &B, plan);
    if (s != DSS_OK) return s;
    if (workspace && workspace_bytes < B.total)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)B.total);
    s = check_device(plan);
    if (s != DSS_OK) return s;
    char* ws = nullptr;
    s = resolve_workspace(plan, workspace, workspace_bytes, B.total, &ws);
    if (s != DSS_OK) return s;
    hipError_t e;

    const Geom& G = B.G;
    const int L = ch.L();
    auto A = [&](int j) { return (float*)(ws + B.a_off[j]); };
    auto Cv = [&](int j) { return (float*)(ws + B.c_off[j]); };
    float* gb[2] = {(float*)(ws + B.g_off[0]), (float*)(ws + B.g_off[1])};
    float* padb = (float*)(ws + B.pad_off);
    float* wpart = (float*)(ws + B.wpart_off);
    Timer T(plan, stream);

    // forward, keeping every layer's convolution output and pool output
    e = T.run("stuff_pack", 0, 0.0, (double)ch.in_c * ((double)H * W + (double)G.D_h * G.D_w) * 4.0, [&] {
        return launch_stuff_pack(DSS_F32, signal, ch.in_c, H, W, A(0), G.D_h, G.D_w, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "stuff_pack launch");
    for (int j = 1; j <= L; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        const LayerGeom& lg = G.L[j - 1];
        const int Fin = lg.Fin_h * lg.Fin_w;
        if (c.has_conv) {
            const PlanConv pc = mfma_launch_variant(plan->convs[j - 1], Fin, lg.Uin_h, lg.Uin_w, 1, 1);
            const double fl = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            e = T.run(conv_name(pc, DSS_F32), j, fl, 0.0, [&]() -> hipError_t {
                if (pc.impl == CONV_MFMA_F32)
                    return launch_conv_mfma_f32(A(j - 1), Fin, lg.Uin_h, lg.Uin_w, 1, 1, pc, Cv(j), stream);
                return launch_conv_direct(DSS_F32, DSS_F32, A(j - 1), Fin, lg.Uin_h, lg.Uin_w, 1, 1, c.cin, pc, Cv(j),
                                          stream);
            });
            if (e != hipSuccess) return hip_fail(e, "conv launch");
        }
        if (c.has_pool) {
            e = T.run("pool_frag", j, 0.0, 0.0, [&] {
                return launch_pool_frag(DSS_F32, Cv(j), lg.Fin_h, lg.Fin_w, lg.E_h, lg.E_w, c.cout, c.k_h, c.k_w, A(j),
                                        stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pool_frag launch");
        }
    }

    // upstream gradient into the final fragment layout (transpose of Defrag + Trim)
    int cur = 0;
    e = T.run("frag_scatter_grad", L + 1, 0.0, 0.0, [&] {
        return launch_frag_scatter_grad(grad_out, ch.out_c(), G.out_h, G.out_w, ch.K_h(), ch.K_w(), G.L.back().U_h,
                                        G.L.back().U_w, gb[cur], stream);
    });
    if (e != hipSuccess) return hip_fail(e, "frag_scatter_grad launch");
    for (int j = L; j >= 1; --j) {
        const ChainLayer& c = ch.layers[j - 1];
        const LayerGeom& lg = G.L[j - 1];
        const int Fin = lg.Fin_h * lg.Fin_w;
        if (c.has_pool) {
            const int act = c.has_conv ? c.act : DSS_ACT_NONE;
            e = T.run("pool_frag_backward", j, 0.0, 0.0, [&] {
                return launch_pool_frag_backward(gb[cur], Cv(j), lg.Fin_h, lg.Fin_w, lg.E_h, lg.E_w, c.cout, c.k_h,
                                                 c.k_w, act, gb[cur ^ 1], stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pool_frag_backward launch");
            cur ^= 1;
        } else if (c.act != DSS_ACT_NONE) {
            const int64_t n = (int64_t)Fin * lg.E_h * lg.E_w * c.cout;
            e = T.run("act_backward", j, 0.0, 0.0,
                      [&] { return launch_act_backward(gb[cur], Cv(j), n, c.act, gb[cur ^ 1], stream); });
            if (e != hipSuccess) return hip_fail(e, "act_backward launch");
            cur ^= 1;
        }
        if (!c.has_conv) continue;   // the pool backward produced the gradient of A_{j-1}
        const double fl = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
        const WgradPlan& wp = B.wg[j];
        e = T.run("wgrad_mfma", j, fl, 0.0, [&] {
            return launch_wgrad(gb[cur], A(j - 1), Fin, lg.E_h, lg.E_w, lg.Uin_h, lg.Uin_w, c.cout, c.cin, c.c_h, c.c_w,
                                wp, wpart, grad_weight + B.wofs[j], grad_bias + B.bofs[j], stream);
        });
        if (e != hipSuccess) return hip_fail(e, "wgrad launch");
        if (j == 1 && !grad_signal) break;
        // input gradient: the full convolution of the output gradient with the
        // transposed, flipped filters, i.e. a valid convolution over the gradient
        // with a zero border of fh - 1 x fw - 1 samples
        const int ph = c.c_h - 1, pw = c.c_w - 1;
        const PlanConv bpc = mfma_launch_variant(plan->bconvs[j - 1], Fin, lg.E_h, lg.E_w, 1, 1, ph, pw);
        if (bpc.impl != CONV_MFMA_F32) {
            e = T.run("pad_grad", j, 0.0, 0.0, [&] {
                return launch_pad_grad(gb[cur], Fin, lg.E_h, lg.E_w, c.cout, ph, pw, padb, stream);
            });
            if (e != hipSuccess) return hip_fail(e, "pad_grad launch");
        }
        const int Hp = lg.E_h + 2 * ph, Wp = lg.E_w + 2 * pw;
        e = T.run(dgrad_name(bpc), j, fl, 0.0, [&]() -> hipError_t {
            if (bpc.impl == CONV_MFMA_F32)
                return launch_conv_mfma_f32_padded(gb[cur], Fin, lg.E_h, lg.E_w, ph, pw, bpc, gb[cur ^ 1], stream);
            return launch_conv_direct(DSS_F32, DSS_F32, padb, Fin, Hp, Wp, 1, 1, c.cout, bpc, gb[cur ^ 1], stream);
        });
        if (e != hipSuccess) return hip_fail(e, "input-gradient conv launch");
        cur ^= 1;
    }
    if (grad_signal) {
        e = T.run("crop_to_planar", 0, 0.0, 0.0,
                  [&] { return launch_crop_to_planar(gb[cur], G.D_w, ch.in_c, H, W, grad_signal, stream); });
        if (e != hipSuccess) return hip_fail(e, "crop_to_planar launch");
    }
    return DSS_OK;
}

// ------------------------------------------------------------------ Frag / Defrag

static dss_status frag_common(bool inverse, int32_t kh, int32_t kw, int32_t Sh, int32_t Sw, int32_t C, int32_t H,
                              int32_t W, dss_dtype dtype, const void* in, void* out, hipStream_t stream) {
    if (!in || !out) return fail(DSS_E_INVALID, "NULL in or out");
    if (dtype != DSS_F32 && dtype != DSS_BF16) return fail(DSS_E_UNSUPPORTED, "unknown dtype %d", dtype);
    if (kh <= 0 || kw <= 0 || Sh <= 0 || Sw <= 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(DSS_E_INVALID, "sizes must be positive");
    if (!inverse && (H % kh != 0 || W % kw != 0))
        return fail(DSS_E_SHAPE, "Frag needs k_h | H and k_w | W (got %dx%d, k %dx%d)", H, W, kh, kw);
    const int64_t n = (int64_t)kh * kw * Sh * Sw * C * H * W;
    if (n > ((int64_t)1 << 40)) return fail(DSS_E_UNSUPPORTED, "tensor too large");
    const size_t es = dtype_size(dtype);
    const char* a = (const char*)in;
    const char* b = (const char*)out;
    const size_t bytes = (size_t)Sh * Sw * C * H * W * es * (inverse ? (size_t)kh * kw : 1);
    if (a < b + bytes && b < a + bytes) return fail(DSS_E_INVALID, "in and out overlap");
    hipError_t e = launch_frag_planar((int)es, inverse, in, kh, kw, Sh, Sw, C, H, W, out, stream);
    if (e != hipSuccess) return hip_fail(e, inverse ? "defrag launch" : "frag launch");
    return DSS_OK;
}

extern "C" dss_status dss_frag(int32_t k_h, int32_t k_w, int32_t S_h, int32_t S_w, int32_t C, int32_t H, int32_t W,
                               dss_dtype dtype, const void* in, void* out, hipStream_t stream) {
    return frag_common(false, k_h, k_w, S_h, S_w, C, H, W, dtype, in, out, stream);
}

extern "C" dss_status dss_defrag(int32_t k_h, int32_t k_w, int32_t S_h, int32_t S_w, int32_t C, int32_t H, int32_t W,
                                 dss_dtype dtype, const void* in, void* out, hipStream_t stream) {
    return frag_common(true, k_h, k_w, S_h, S_w, C, H, W, dtype, in, out, stream);
}
