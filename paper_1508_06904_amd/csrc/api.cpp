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
static ConvImpl choose_impl(const ChainLayer& c, dss_dtype dt) {
    // Tuning / cross-check override: DSS_CONV_KERNEL=direct selects the VALU
    // kernel for every convolution of plans created afterwards.
    const char* force = getenv("DSS_CONV_KERNEL");
    if (force && std::strcmp(force, "direct") == 0) return CONV_DIRECT;
    if (c.cin < 16) return CONV_DIRECT;
    if (dt == DSS_F32 && c.cin % 4 == 0 && mfma_supports(false, c.cout, c.c_h, c.c_w)) return CONV_MFMA_F32;
    if (dt == DSS_BF16 && c.cin % 8 == 0 && mfma_supports(true, c.cout, c.c_h, c.c_w)) return CONV_MFMA_BF16;
    return CONV_DIRECT;
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
    for (auto& c : p->convs) {
        if (c.w) (void)hipFree(c.w);
        if (c.b) (void)hipFree(c.b);
        c.w = nullptr;
        c.b = nullptr;
    }
    for (hipEvent_t e : p->events) (void)hipEventDestroy(e);
    p->events.clear();
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
    for (int j = 0; j < L; ++j) {
        const ChainLayer& c = p->chain.layers[j];
        if (!c.has_conv) continue;
        const dss_layer& d = layers[c.desc];
        PlanConv& pc = p->convs[j];
        pc.cin = c.cin;
        pc.cout = c.cout;
        pc.fh = c.c_h;
        pc.fw = c.c_w;
        pc.act = c.act;
        pc.impl = choose_impl(c, dtype);
        const bool bf16 = dtype == DSS_BF16;
        std::vector<float> bias;
        std::vector<char> wbuf;
        size_t wbytes = 0;
        if (pc.impl == CONV_DIRECT) {
            // [fh][fw][cin][cout_pad] binary32 (bfloat16-rounded values for bfloat16 plans)
            pc.cob = c.cout >= 16 ? 16 : c.cout >= 8 ? 8 : c.cout >= 4 ? 4 : c.cout >= 2 ? 2 : 1;
            pc.cout_pad = (c.cout + pc.cob - 1) / pc.cob * pc.cob;
            wbytes = sizeof(float) * (size_t)pc.fh * pc.fw * pc.cin * pc.cout_pad;
            wbuf.assign(wbytes, 0);
            float* w = reinterpret_cast<float*>(wbuf.data());
            for (int o = 0; o < c.cout; ++o)
                for (int i = 0; i < c.cin; ++i)
                    for (int th = 0; th < pc.fh; ++th)
                        for (int tw = 0; tw < pc.fw; ++tw) {
                            float v = d.weight[(((size_t)o * c.cin + i) * pc.fh + th) * pc.fw + tw];
                            if (bf16) {
                                const uint32_t u = (uint32_t)host_f32_to_bf16(v) << 16;
                                std::memcpy(&v, &u, 4);
                            }
                            w[(((size_t)th * pc.fw + tw) * pc.cin + i) * pc.cout_pad + o] = v;
                        }
            bias.assign(pc.cout_pad, 0.f);
        } else if (pc.impl == CONV_MFMA_F32) {
            pc.bn = mfma_f32_pick_bn(c.cout);
            pc.cin_pad = (c.cin + 15) / 16 * 16;
            pc.cout_pad = (c.cout + pc.bn - 1) / pc.bn * pc.bn;
            wbytes = sizeof(float) * mfma_f32_packed_floats(pc);
            wbuf.assign(wbytes, 0);
            mfma_f32_pack(pc, d.weight, reinterpret_cast<float*>(wbuf.data()));
            bias.assign(pc.cout_pad, 0.f);
        } else {
            pc.bn = mfma_bf16_pick_bn(c.cout);
            pc.cin_pad = (c.cin + 31) / 32 * 32;
            pc.cout_pad = (c.cout + pc.bn - 1) / pc.bn * pc.bn;
            wbytes = sizeof(uint16_t) * mfma_bf16_packed_elems(pc);
            wbuf.assign(wbytes, 0);
            mfma_bf16_pack(pc, d.weight, reinterpret_cast<uint16_t*>(wbuf.data()));
            bias.assign(pc.cout_pad, 0.f);
        }
        for (int o = 0; o < c.cout; ++o) bias[o] = d.bias ? d.bias[o] : 0.f;
        e = hipMalloc(&pc.w, wbytes);
        if (e == hipSuccess) e = hipMalloc((void**)&pc.b, sizeof(float) * bias.size());
        if (e == hipSuccess) e = hipMemcpy(pc.w, wbuf.data(), wbytes, hipMemcpyHostToDevice);
        if (e == hipSuccess) e = hipMemcpy(pc.b, bias.data(), sizeof(float) * bias.size(), hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            s = hip_fail(e, "uploading weights");
            free_plan_memory(p);
            delete p;
            return s;
        }
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
        records[i].reserved = 0;
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
    Timer(dss_plan* p_, hipStream_t s_) : p(p_), s(s_), on(p_->timing) { next = 2 * (int)p->recs.size(); }
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
    hipError_t run(const char* name, int layer, double flops, double bytes, F&& launch) {
        if (!on) return launch();
        LaunchRec r{name, layer, flops, bytes, 0, 0};
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
            return "conv_direct";
    }
}

}  // namespace

// Runs Stuff and chain layers 1..upto.  On return *cur points at the last
// tensor (channels-last fragment layout) and *cur_dt is its element type.
// Chain layers 1..upto on the packed input in buf[0] (the two halves of the
// workspace ping-pong).  On return *cur points at the last tensor (channels-last
// fragment layout) and *cur_dt is its element type.  A relaxed layer's pooling
// runs over all Fin fragments at once as one tall signal of Fin * E_h rows:
// every fragment's extent is a multiple of k_h, so no block straddles two.
static dss_status run_layers(dss_plan* p, const Geom& G, int upto, char* const buf[2], hipStream_t stream, Timer& T,
                             void** cur_out, dss_dtype* cur_dt) {
    const Chain& ch = p->chain;
    int which = 0;
    const dss_dtype dt = p->dtype;
    const double es = (double)dtype_size(dt);
    hipError_t e;
    void* cur = buf[0];
    dss_dtype cdt = dt;
    for (int j = 1; j <= upto; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        const LayerGeom& lg = G.L[j - 1];
        const int Fin = lg.Fin_h * lg.Fin_w;
        if (c.has_conv) {
            const PlanConv& pc = p->convs[j - 1];
            const bool last_op = (j == ch.L()) && !c.has_pool;
            const dss_dtype tout = (dt == DSS_BF16 && last_op) ? DSS_F32 : dt;
            void* dst = buf[which ^ 1];
            const double flops = 2.0 * Fin * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const double bytes = (double)Fin * lg.Uin_h * lg.Uin_w * c.cin * dtype_size(cdt) +
                                 (double)Fin * lg.E_h * lg.E_w * c.cout * dtype_size(tout) +
                                 (double)c.cout * c.cin * c.c_h * c.c_w * es;
            e = T.run(conv_name(pc, tout), j, flops, bytes, [&]() -> hipError_t {
                if (pc.impl == CONV_MFMA_F32)
                    return launch_conv_mfma_f32((const float*)cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w, pc,
                                                (float*)dst, stream);
                if (pc.impl == CONV_MFMA_BF16)
                    return launch_conv_mfma_bf16(tout, (const uint16_t*)cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h,
                                                 lg.dil_w, pc, dst, stream);
                return launch_conv_direct(cdt, tout, cur, Fin, lg.Uin_h, lg.Uin_w, lg.dil_h, lg.dil_w, c.cin, pc, dst,
                                          stream);
            });
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
                            hipStream_t stream, Timer& T, void** cur_out, dss_dtype* cur_dt) {
    const Chain& ch = p->chain;
    char* const buf[2] = {ws, ws + G.buf_bytes};
    const dss_dtype dt = p->dtype;
    const double es = (double)dtype_size(dt);
    const double in_read = (double)std::min(G.H, G.D_h) * std::min(G.W, G.D_w);
    hipError_t e = T.run("stuff_pack", 0, 0.0, (double)ch.in_c * (in_read + G.D_h * (double)G.D_w) * es,
                         [&] { return launch_stuff_pack(dt, signal, ch.in_c, G.H, G.W, buf[0], G.D_h, G.D_w, stream); });
    if (e != hipSuccess) return hip_fail(e, "stuff_pack launch");
    return run_layers(p, G, upto, buf, stream, T, cur_out, cur_dt);
}

static dss_status check_eval_args(dss_plan_t plan, const void* signal, const void* out, void* workspace,
                                  int64_t workspace_bytes, int32_t H, int32_t W, int32_t ell, Geom* G) {
    if (!plan || !signal || !out) return fail(DSS_E_INVALID, "NULL plan, signal or out");
    dss_status s = compute_geometry(plan->chain, plan->dtype, H, W, ell, G);
    if (s != DSS_OK) return s;
    if (!workspace) return fail(DSS_E_INVALID, "NULL workspace (need %lld bytes)", (long long)G->ws_bytes);
    if (workspace_bytes < G->ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G->ws_bytes);
    if (((uintptr_t)workspace & 255u) != 0) return fail(DSS_E_INVALID, "workspace is not 256-byte aligned");
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != plan->device)
        return fail(DSS_E_INVALID, "plan belongs to device %d but device %d is current", plan->device, cur);
    return DSS_OK;
}

extern "C" dss_status dss_eval_mixed(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                                     float* out, void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    Geom G;
    dss_status s = check_eval_args(plan, signal, out, workspace, workspace_bytes, H, W, ell, &G);
    if (s != DSS_OK) return s;
    Timer T(plan, stream);
    void* cur = nullptr;
    dss_dtype cdt;
    s = run_chain(plan, G, signal, plan->chain.L(), (char*)workspace, stream, T, &cur, &cdt);
    if (s != DSS_OK) return s;
    const Chain& ch = plan->chain;
    // Defrag_{k*_L / k*_ell}, then keep the first out_h x out_w samples (this is
    // Trim_r of the dense evaluation and the final trimming of the stuffing mode)
    const int Gh = ch.K_h() / G.step_h, Gw = ch.K_w() / G.step_w;
    const int Uh = G.L.back().U_h, Uw = G.L.back().U_w;
    const double bytes = (double)Gh * Gw * Uh * Uw * ch.out_c() * dtype_size(cdt) +
                         (double)G.out_h * G.out_w * ch.out_c() * 4.0;
    hipError_t e = T.run("defrag_trim", ch.L() + 1, 0.0, bytes, [&] {
        return launch_defrag_trim(cdt, cur, Gh, Gw, Uh, Uw, ch.out_c(), out, G.out_h, G.out_w, stream);
    });
    if (e != hipSuccess) return hip_fail(e, "defrag_trim launch");
    return DSS_OK;
}

extern "C" dss_status dss_eval_dense(dss_plan_t plan, const void* signal, int32_t H, int32_t W, float* out,
                                     void* workspace, int64_t workspace_bytes, hipStream_t stream) {
    return dss_eval_mixed(plan, signal, H, W, 0, out, workspace, workspace_bytes, stream);
}

extern "C" dss_status dss_eval_slide(dss_plan_t plan, const void* signal, int32_t H, int32_t W, int32_t ell,
                                     int32_t j, float* out, void* workspace, int64_t workspace_bytes,
                                     hipStream_t stream) {
    Geom G;
    dss_status s = check_eval_args(plan, signal, out, workspace, workspace_bytes, H, W, ell, &G);
    if (s != DSS_OK) return s;
    if (j < 0 || j > plan->chain.L()) return fail(DSS_E_INVALID, "chain layer %d out of range 0..%d", j, plan->chain.L());
    Timer T(plan, stream);
    void* cur = nullptr;
    dss_dtype cdt;
    s = run_chain(plan, G, signal, j, (char*)workspace, stream, T, &cur, &cdt);
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
    if (!workspace) return fail(DSS_E_INVALID, "NULL workspace (need %lld bytes)", (long long)G.ws_bytes);
    if (workspace_bytes < G.ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G.ws_bytes);
    if (((uintptr_t)workspace & 255u) != 0) return fail(DSS_E_INVALID, "workspace is not 256-byte aligned");
    int cur_dev = -1;
    hipError_t e = hipGetDevice(&cur_dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur_dev != plan->device)
        return fail(DSS_E_INVALID, "plan belongs to device %d but device %d is current", plan->device, cur_dev);

    Timer T(plan, stream);
    char* const buf[2] = {(char*)workspace, (char*)workspace + G.buf_bytes};
    const double es = (double)dtype_size(plan->dtype);
    const double pbytes = 2.0 * count * (double)ch.B_h * ch.B_w * ch.in_c * es;
    e = T.run("patch_pack", 0, 0.0, pbytes, [&] {
        return launch_patch_pack(plan->dtype, signal, ch.in_c, H, W, O_w, first, count, ch.B_h, ch.B_w, buf[0],
                                 stream);
    });
    if (e != hipSuccess) return hip_fail(e, "patch_pack launch");
    void* cur = nullptr;
    dss_dtype cdt;
    s = run_layers(plan, G, ch.L(), buf, stream, T, &cur, &cdt);
    if (s != DSS_OK) return s;
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
    if (!workspace) return fail(DSS_E_INVALID, "NULL workspace (need %lld bytes)", (long long)G.ws_bytes);
    if (workspace_bytes < G.ws_bytes)
        return fail(DSS_E_SHAPE, "workspace of %lld bytes is smaller than the %lld bytes needed",
                    (long long)workspace_bytes, (long long)G.ws_bytes);
    if (((uintptr_t)workspace & 255u) != 0) return fail(DSS_E_INVALID, "workspace is not 256-byte aligned");
    int cur_dev = -1;
    hipError_t e = hipGetDevice(&cur_dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur_dev != plan->device)
        return fail(DSS_E_INVALID, "plan belongs to device %d but device %d is current", plan->device, cur_dev);
    Timer T(plan, stream);
    void* cur = nullptr;
    dss_dtype cdt;
    s = run_chain(plan, G, signal, j, (char*)workspace, stream, T, &cur, &cdt);   // D = H x W: a plain pack
    if (s != DSS_OK) return s;
    const int h = j == 0 ? H : G.L[j - 1].U_h;
    const int w = j == 0 ? W : G.L[j - 1].U_w;
    const int C = j == 0 ? ch.in_c : ch.layers[j - 1].cout;
    const double bytes = (double)h * w * C * (dtype_size(cdt) + 4.0);
    e = T.run("to_planar", ch.L() + 1, 0.0, bytes, [&] { return launch_to_planar(cdt, cur, 1, h, w, C, out, stream); });
    if (e != hipSuccess) return hip_fail(e, "to_planar launch");
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
