// Processing chain and per-signal geometry (host only, integer arithmetic).
//
//  * Grouping of the layer list into processing-chain layers: a convolution and
//    the max-pool that directly follows it form one layer; a convolution without
//    a pool gets k = 1 and a pool without a convolution gets the identity
//    transformation c = 1 (bypass layers, end of Sect. 4.2).
//  * Receptive field and stride products (Definition "processing chain" and
//    Lemma "processing chain" (a), Sect. 4.2): starting from u_L = 1 the strided
//    extents satisfy u_{j-1} - c_j + 1 = k_j u_j (Sect. 5.1), so
//    B = u_0 and k*_j = k_1 ... k_j.
//  * Stuffing count r = 0 if k*_L divides N - B + 1, else k*_L - rem(N - B + 1, k*_L)
//    (Theorem "processing chain", Sect. 4.3), per axis.  At a mixed level
//    ell > 0 the operating modes of Theorem "evalrelaxslide" (appendix) trim or
//    stuff instead; ell = 0 is the case above.
//  * Fragment extents of the sliding evaluation: U_0 = D = N + r, after T_j the
//    extent is U_{j-1} - c_j + 1, after Slide_g it is one sample shorter per
//    extra pooled sample, and Frag_k divides it by k (Lemma (b)); the fragment
//    count per axis is k*_j (k*_j / k*_ell after ell relaxed layers, which keep
//    one fragment and divide the extent by k_j: Lemma "evalrelax" (b)).
#include <algorithm>
#include <cstring>

#include "dss_internal.h"

namespace dss {

size_t dtype_size(dss_dtype dt) { return dt == DSS_BF16 ? 2 : 4; }

dss_status build_chain(const dss_layer* layers, int n, int ndim, int in_c, Chain* out) {
    if (!layers || n <= 0) return fail(DSS_E_INVALID, "empty layer list");
    if (ndim != 1 && ndim != 2) return fail(DSS_E_UNSUPPORTED, "ndim must be 1 or 2 (got %d)", ndim);
    if (in_c <= 0) return fail(DSS_E_INVALID, "in_channels must be positive (got %d)", in_c);
    Chain ch;
    ch.ndim = ndim;
    ch.in_c = in_c;
    int cur_c = in_c;
    int t = 0;
    while (t < n) {
        const dss_layer& l = layers[t];
        ChainLayer cl;
        if (l.kind == DSS_LAYER_CONV) {
            if (l.cin != cur_c)
                return fail(DSS_E_INVALID, "layer %d: cin=%d but the previous layer gives %d channels", t, l.cin, cur_c);
            if (l.cout <= 0 || l.fh <= 0 || l.fw <= 0)
                return fail(DSS_E_INVALID, "layer %d: non-positive conv size", t);
            if (ndim == 1 && l.fh != 1) return fail(DSS_E_INVALID, "layer %d: 1-D networks need fh = 1", t);
            if (l.act < DSS_ACT_NONE || l.act > DSS_ACT_TANH)
                return fail(DSS_E_INVALID, "layer %d: unknown activation %d", t, l.act);
            if (!l.weight) return fail(DSS_E_INVALID, "layer %d: NULL weight", t);
            cl.has_conv = true;
            cl.c_h = l.fh;
            cl.c_w = l.fw;
            cl.cin = l.cin;
            cl.cout = l.cout;
            cl.act = l.act;
            cl.desc = t;
            cur_c = l.cout;
            ++t;
            if (t < n && layers[t].kind == DSS_LAYER_MAXPOOL) {
                const dss_layer& p = layers[t];
                if (p.kh <= 0 || p.kw <= 0) return fail(DSS_E_INVALID, "layer %d: non-positive pool size", t);
                if (ndim == 1 && p.kh != 1) return fail(DSS_E_INVALID, "layer %d: 1-D networks need kh = 1", t);
                cl.has_pool = true;
                cl.k_h = p.kh;
                cl.k_w = p.kw;
                ++t;
            }
        } else if (l.kind == DSS_LAYER_MAXPOOL) {
            if (l.kh <= 0 || l.kw <= 0) return fail(DSS_E_INVALID, "layer %d: non-positive pool size", t);
            if (ndim == 1 && l.kh != 1) return fail(DSS_E_INVALID, "layer %d: 1-D networks need kh = 1", t);
            cl.has_pool = true;
            cl.k_h = l.kh;
            cl.k_w = l.kw;
            cl.cin = cl.cout = cur_c;
            ++t;
        } else {
            return fail(DSS_E_INVALID, "layer %d: unknown kind %d", t, l.kind);
        }
        ch.layers.push_back(cl);
    }
    const int L = ch.L();
    ch.kstar_h.assign(L + 1, 1);
    ch.kstar_w.assign(L + 1, 1);
    for (int j = 1; j <= L; ++j) {
        const int64_t kh = (int64_t)ch.kstar_h[j - 1] * ch.layers[j - 1].k_h;
        const int64_t kw = (int64_t)ch.kstar_w[j - 1] * ch.layers[j - 1].k_w;
        if (kh > (1 << 20) || kw > (1 << 20)) return fail(DSS_E_UNSUPPORTED, "stride product too large");
        ch.kstar_h[j] = (int)kh;
        ch.kstar_w[j] = (int)kw;
    }
    ch.u_h.assign(L + 1, 1);
    ch.u_w.assign(L + 1, 1);
    for (int j = L; j >= 1; --j) {
        const ChainLayer& c = ch.layers[j - 1];
        const int64_t uh = (int64_t)c.k_h * ch.u_h[j] + c.c_h - 1;
        const int64_t uw = (int64_t)c.k_w * ch.u_w[j] + c.c_w - 1;
        if (uh > (1 << 28) || uw > (1 << 28)) return fail(DSS_E_UNSUPPORTED, "receptive field too large");
        ch.u_h[j - 1] = (int)uh;
        ch.u_w[j - 1] = (int)uw;
    }
    ch.B_h = ch.u_h[0];
    ch.B_w = ch.u_w[0];
    *out = std::move(ch);
    return DSS_OK;
}

// Operating mode per axis (Theorem "evalrelaxslide"; for k = 1 it reduces to the
// stuffing of Theorem "processing chain", for k = K to the trimming of Theorem
// "evalrelax"): r = rem(N - B + k, K) with k = k*_ell and K = k*_L; trim r
// samples if r < k, else stuff K - r.
static void operating_mode(int N, int B, int K, int k, int* trim, int* stuff) {
    const int r = (int)(((int64_t)N - B + k) % K);
    *trim = r < k ? r : 0;
    *stuff = r < k ? 0 : K - r;
}

dss_status compute_geometry(const Chain& ch, dss_dtype dt, int H, int W, int ell, Geom* g) {
    if (ch.ndim == 1 && H != 1) return fail(DSS_E_SHAPE, "1-D plan needs H = 1 (got %d)", H);
    if (H < ch.B_h || W < ch.B_w)
        return fail(DSS_E_SHAPE, "signal %dx%d is smaller than the receptive field %dx%d", H, W, ch.B_h, ch.B_w);
    const int L = ch.L();
    if (ell < 0 || ell > L) return fail(DSS_E_INVALID, "mixed level %d out of range 0..%d", ell, L);
    Geom G;
    G.ell = ell;
    G.step_h = ch.kstar_h[ell];
    G.step_w = ch.kstar_w[ell];
    G.H = H;
    G.W = W;
    operating_mode(H, ch.B_h, ch.K_h(), G.step_h, &G.trim_h, &G.r_h);
    operating_mode(W, ch.B_w, ch.K_w(), G.step_w, &G.trim_w, &G.r_w);
    G.D_h = H - G.trim_h + G.r_h;
    G.D_w = W - G.trim_w + G.r_w;
    G.out_h = (H - ch.B_h) / G.step_h + 1;   // ceil((H - B + 1) / k*_ell)
    G.out_w = (W - ch.B_w) / G.step_w + 1;
    // Lemma "evalrelaxslide": D = B + k*_L t - k*_ell with t >= 1
    const int64_t th = ((int64_t)G.D_h - ch.B_h + G.step_h) / ch.K_h();
    const int64_t tw = ((int64_t)G.D_w - ch.B_w + G.step_w) / ch.K_w();
    if (th < 1 || tw < 1 || th * ch.K_h() != (int64_t)G.D_h - ch.B_h + G.step_h ||
        tw * ch.K_w() != (int64_t)G.D_w - ch.B_w + G.step_w)
        return fail(DSS_E_SHAPE, "trimmed/stuffed extents %dx%d violate the divisibility requirement", G.D_h, G.D_w);
    const double es = (double)dtype_size(dt);

    int Uh = G.D_h, Uw = G.D_w;
    int cur_c = ch.in_c;
    int64_t maxbuf = (int64_t)G.D_h * G.D_w * ch.in_c * (int64_t)es;
    G.total_bytes = (double)ch.in_c * std::min(H, G.D_h) * std::min(W, G.D_w) * es +
                    (double)ch.in_c * G.D_h * G.D_w * es;
    for (int j = 1; j <= L; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        LayerGeom lg;
        lg.relaxed = j <= ell;
        lg.Uin_h = Uh;
        lg.Uin_w = Uw;
        lg.Fin_h = lg.relaxed ? 1 : ch.kstar_h[j - 1] / G.step_h;
        lg.Fin_w = lg.relaxed ? 1 : ch.kstar_w[j - 1] / G.step_w;
        lg.Fout_h = lg.relaxed ? 1 : ch.kstar_h[j] / G.step_h;
        lg.Fout_w = lg.relaxed ? 1 : ch.kstar_w[j] / G.step_w;
        const int64_t Fin = (int64_t)lg.Fin_h * lg.Fin_w;
        lg.E_h = Uh - c.c_h + 1;
        lg.E_w = Uw - c.c_w + 1;
        if (lg.E_h < c.k_h || lg.E_w < c.k_w) return fail(DSS_E_SHAPE, "layer %d: extent underflow", j);
        if (lg.relaxed) {
            // Stride_g: non-overlapping blocks
            if (lg.E_h % c.k_h != 0 || lg.E_w % c.k_w != 0)
                return fail(DSS_E_SHAPE, "layer %d: relaxed extent %dx%d not divisible by %dx%d", j, lg.E_h, lg.E_w,
                            c.k_h, c.k_w);
            lg.U_h = lg.E_h / c.k_h;
            lg.U_w = lg.E_w / c.k_w;
        } else {
            const int Ph = lg.E_h - c.k_h + 1, Pw = lg.E_w - c.k_w + 1;
            if (Ph % c.k_h != 0 || Pw % c.k_w != 0)
                return fail(DSS_E_SHAPE, "layer %d: sliding-pool extent %dx%d not divisible by %dx%d", j, Ph, Pw,
                            c.k_h, c.k_w);
            lg.U_h = Ph / c.k_h;
            lg.U_w = Pw / c.k_w;
        }
        // the final conv of a bfloat16 plan stores binary32
        const bool last_op = (j == L) && !c.has_pool;
        if (c.has_conv) {
            const double es_out = (dt == DSS_BF16 && last_op) ? 4.0 : es;
            const double macs = (double)Fin * lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            G.conv_flops += 2.0 * macs;
            const int64_t out_b = Fin * lg.E_h * lg.E_w * c.cout * (int64_t)es_out;
            maxbuf = std::max(maxbuf, out_b);
            G.total_bytes += (double)Fin * Uh * Uw * c.cin * es + (double)out_b +
                             (double)c.cout * c.cin * c.c_h * c.c_w * (dt == DSS_BF16 ? 2.0 : 4.0);
        }
        if (c.has_pool) {
            const int64_t Fout = (int64_t)lg.Fout_h * lg.Fout_w;
            const double pb = (double)Fin * lg.E_h * lg.E_w * c.cout * es + (double)Fout * lg.U_h * lg.U_w * c.cout * es;
            G.pool_bytes += pb;
            G.total_bytes += pb;
            maxbuf = std::max(maxbuf, Fout * lg.U_h * lg.U_w * c.cout * (int64_t)es);
        }
        if (lg.relaxed) {
            // Lemma "evalrelax" (b): W_j - u_j = (D - B) / k*_j
            if ((int64_t)(lg.U_h - ch.u_h[j]) * ch.kstar_h[j] != (int64_t)G.D_h - ch.B_h ||
                (int64_t)(lg.U_w - ch.u_w[j]) * ch.kstar_w[j] != (int64_t)G.D_w - ch.B_w)
                return fail(DSS_E_SHAPE, "layer %d: relaxed extent disagrees with Lemma \"evalrelax\" (b)", j);
        } else {
            // Lemma "evalrelaxslide" (b) (Lemma "processing chain" (b) for ell = 0):
            // U_j - u_j + 1 = (k*_L / k*_j) t
            if ((int64_t)(lg.U_h - ch.u_h[j] + 1) * ch.kstar_h[j] != th * ch.K_h() ||
                (int64_t)(lg.U_w - ch.u_w[j] + 1) * ch.kstar_w[j] != tw * ch.K_w())
                return fail(DSS_E_SHAPE, "layer %d: fragment extent disagrees with Lemma (b)", j);
        }
        G.L.push_back(lg);
        Uh = lg.U_h;
        Uw = lg.U_w;
        cur_c = c.cout;
    }
    // After Defrag_{k*_L / k*_ell} there are (k*_L / k*_ell) t = (D - B)/k*_ell + 1
    // samples per axis; the output keeps the first ceil((N - B + 1)/k*_ell).
    const int Gh = ch.K_h() / G.step_h, Gw = ch.K_w() / G.step_w;
    if ((int64_t)Uh * Gh < G.out_h || (int64_t)Uw * Gw < G.out_w)
        return fail(DSS_E_SHAPE, "final fragment extent is smaller than the output");
    const bool last_f32 = dt == DSS_BF16 && !ch.layers.back().has_pool && ch.layers.back().has_conv;
    const double es_last = last_f32 ? 4.0 : es;
    G.total_bytes += (double)Gh * Gw * Uh * Uw * cur_c * es_last + (double)G.out_h * G.out_w * cur_c * 4.0;
    G.buf_bytes = (maxbuf + 255) / 256 * 256;
    G.ws_bytes = 2 * G.buf_bytes;
    *g = std::move(G);
    return DSS_OK;
}

// The strided network on a batch of `count` windows (EvalStride of Definition
// "processing chain", Sect. 4.2): each window is a fragment of B_h x B_w samples,
// every layer is relaxed (conv on each fragment, then max-pool with stride k_j),
// and after layer j each fragment holds u_j samples per axis (Lemma (a)).
dss_status compute_stride_geometry(const Chain& ch, dss_dtype dt, int count, Geom* g) {
    if (count <= 0) return fail(DSS_E_INVALID, "window count must be positive (got %d)", count);
    const int L = ch.L();
    Geom G;
    G.ell = L;
    G.H = G.D_h = ch.B_h;
    G.W = G.D_w = ch.B_w;
    G.out_h = G.out_w = 1;
    G.step_h = ch.K_h();
    G.step_w = ch.K_w();
    const double es = (double)dtype_size(dt);
    int Uh = ch.B_h, Uw = ch.B_w;
    int64_t maxbuf = (int64_t)count * Uh * Uw * ch.in_c * (int64_t)es;
    G.total_bytes = 2.0 * (double)count * Uh * Uw * ch.in_c * es;
    for (int j = 1; j <= L; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        LayerGeom lg;
        lg.relaxed = true;
        lg.Uin_h = Uh;
        lg.Uin_w = Uw;
        lg.Fin_h = lg.Fout_h = count;
        lg.Fin_w = lg.Fout_w = 1;
        lg.E_h = Uh - c.c_h + 1;
        lg.E_w = Uw - c.c_w + 1;
        lg.U_h = lg.E_h / c.k_h;
        lg.U_w = lg.E_w / c.k_w;
        if (lg.U_h != ch.u_h[j] || lg.U_w != ch.u_w[j] || lg.E_h != c.k_h * ch.u_h[j] || lg.E_w != c.k_w * ch.u_w[j])
            return fail(DSS_E_SHAPE, "layer %d: strided extents disagree with Lemma (a)", j);
        const bool last_op = (j == L) && !c.has_pool;
        if (c.has_conv) {
            const double es_out = (dt == DSS_BF16 && last_op) ? 4.0 : es;
            G.conv_flops += 2.0 * (double)count * lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const int64_t out_b = (int64_t)count * lg.E_h * lg.E_w * c.cout * (int64_t)es_out;
            maxbuf = std::max(maxbuf, out_b);
            G.total_bytes += (double)count * Uh * Uw * c.cin * es + (double)out_b +
                             (double)c.cout * c.cin * c.c_h * c.c_w * (dt == DSS_BF16 ? 2.0 : 4.0);
        }
        if (c.has_pool) {
            const double pb = (double)count * ((double)lg.E_h * lg.E_w + (double)lg.U_h * lg.U_w) * c.cout * es;
            G.pool_bytes += pb;
            G.total_bytes += pb;
            maxbuf = std::max(maxbuf, (int64_t)count * lg.U_h * lg.U_w * c.cout * (int64_t)es);
        }
        G.L.push_back(lg);
        Uh = lg.U_h;
        Uw = lg.U_w;
    }
    G.buf_bytes = (maxbuf + 255) / 256 * 256;
    G.ws_bytes = 2 * G.buf_bytes;
    *g = std::move(G);
    return DSS_OK;
}

// The dilated fashion (appendix, Definition "evaldilate"): layer j applies the
// convolution and the pooling kernel with their taps k*_{j-1} samples apart, on
// one signal; no stuffing.  Extents per axis: E_j = V_{j-1} - k*_{j-1}(c_j - 1),
// V_j = E_j - k*_{j-1}(k_j - 1), checked against Lemma "evaldilate" (a), (b).
dss_status compute_dilate_geometry(const Chain& ch, dss_dtype dt, int H, int W, Geom* g) {
    if (ch.ndim == 1 && H != 1) return fail(DSS_E_SHAPE, "1-D plan needs H = 1 (got %d)", H);
    if (H < ch.B_h || W < ch.B_w)
        return fail(DSS_E_SHAPE, "signal %dx%d is smaller than the receptive field %dx%d", H, W, ch.B_h, ch.B_w);
    const int L = ch.L();
    Geom G;
    G.H = G.D_h = H;
    G.W = G.D_w = W;
    G.out_h = H - ch.B_h + 1;
    G.out_w = W - ch.B_w + 1;
    const double es = (double)dtype_size(dt);
    int Vh = H, Vw = W;
    int64_t maxbuf = (int64_t)H * W * ch.in_c * (int64_t)es;
    G.total_bytes = 2.0 * (double)H * W * ch.in_c * es;
    int64_t sum_h = 0, sum_w = 0;
    for (int j = 1; j <= L; ++j) {
        const ChainLayer& c = ch.layers[j - 1];
        LayerGeom lg;
        lg.dilated = true;
        lg.dil_h = ch.kstar_h[j - 1];
        lg.dil_w = ch.kstar_w[j - 1];
        lg.Uin_h = Vh;
        lg.Uin_w = Vw;
        lg.Fin_h = lg.Fin_w = lg.Fout_h = lg.Fout_w = 1;
        lg.E_h = Vh - lg.dil_h * (c.c_h - 1);
        lg.E_w = Vw - lg.dil_w * (c.c_w - 1);
        lg.U_h = lg.E_h - lg.dil_h * (c.k_h - 1);
        lg.U_w = lg.E_w - lg.dil_w * (c.k_w - 1);
        sum_h += (int64_t)ch.kstar_h[j - 1] * (c.c_h + c.k_h - 2);
        sum_w += (int64_t)ch.kstar_w[j - 1] * (c.c_w + c.k_w - 2);
        if (lg.U_h != (int64_t)H - sum_h || lg.U_w != (int64_t)W - sum_w ||
            (int64_t)lg.U_h - (int64_t)ch.kstar_h[j] * (ch.u_h[j] - 1) != (int64_t)H - ch.B_h + 1 ||
            (int64_t)lg.U_w - (int64_t)ch.kstar_w[j] * (ch.u_w[j] - 1) != (int64_t)W - ch.B_w + 1)
            return fail(DSS_E_SHAPE, "layer %d: dilated extents disagree with Lemma \"evaldilate\"", j);
        const bool last_op = (j == L) && !c.has_pool;
        if (c.has_conv) {
            const double es_out = (dt == DSS_BF16 && last_op) ? 4.0 : es;
            G.conv_flops += 2.0 * (double)lg.E_h * lg.E_w * c.cout * (double)c.cin * c.c_h * c.c_w;
            const int64_t out_b = (int64_t)lg.E_h * lg.E_w * c.cout * (int64_t)es_out;
            maxbuf = std::max(maxbuf, out_b);
            G.total_bytes += (double)Vh * Vw * c.cin * es + (double)out_b +
                             (double)c.cout * c.cin * c.c_h * c.c_w * (dt == DSS_BF16 ? 2.0 : 4.0);
        }
        if (c.has_pool) {
            const double pb = ((double)lg.E_h * lg.E_w + (double)lg.U_h * lg.U_w) * c.cout * es;
            G.pool_bytes += pb;
            G.total_bytes += pb;
            maxbuf = std::max(maxbuf, (int64_t)lg.U_h * lg.U_w * c.cout * (int64_t)es);
        }
        G.L.push_back(lg);
        Vh = lg.U_h;
        Vw = lg.U_w;
    }
    G.total_bytes += (double)Vh * Vw * ch.out_c() * 4.0;
    G.buf_bytes = (maxbuf + 255) / 256 * 256;
    G.ws_bytes = 2 * G.buf_bytes;
    *g = std::move(G);
    return DSS_OK;
}

}  // namespace dss
