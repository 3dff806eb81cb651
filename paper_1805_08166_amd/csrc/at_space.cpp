// Host-side construction of schedule spaces (Section 2: multi-level tiling of
// each loop axis, thread binding of the outer bands, unrolling annotations).
//
// A space is summarised for the kernels by a SpaceDesc: the knob sizes and
// mixed-radix weights, the ordered split choices of each axis packed four
// 16-bit factors to a word, and the weight of every axis in every buffer's
// flattened index.  The loop order itself is fixed per template inside the
// feature kernels.
#include <algorithm>
#include <cstring>

#include "at_internal.h"

namespace at {
namespace {

std::vector<int64_t> divisors_of(int64_t n) {
    std::vector<int64_t> d;
    for (int64_t f = 1; f * f <= n; ++f) {
        if (n % f) continue;
        d.push_back(f);
        if (f != n / f) d.push_back(n / f);
    }
    std::sort(d.begin(), d.end());
    return d;
}

// Ordered `levels`-factor splits of n in lexicographic order of
// (f_outer, ..., f_inner), each packed as 16-bit fields, outer level in the
// lowest field; unused fields hold 1.
void append_splits(int64_t n, int levels, std::vector<uint64_t>& out) {
    std::vector<int64_t> f(levels, 1);
    // depth-first walk; at each level take divisors of the remaining extent
    // in ascending order, the last level takes the remainder
    struct Frame { int64_t rest; std::vector<int64_t> divs; size_t next; };
    std::vector<Frame> stack;
    stack.push_back(Frame{n, divisors_of(n), 0});
    while (!stack.empty()) {
        int lvl = (int)stack.size() - 1;
        Frame& fr = stack.back();
        if (lvl == levels - 1) {
            f[lvl] = fr.rest;
            uint64_t w = 0;
            for (int l = 0; l < 4; ++l) w |= (uint64_t)(l < levels ? f[l] : 1) << (16 * l);
            out.push_back(w);
            stack.pop_back();
            continue;
        }
        if (fr.next == fr.divs.size()) {
            stack.pop_back();
            continue;
        }
        int64_t d = fr.divs[fr.next++];
        f[lvl] = d;
        int64_t rest = fr.rest / d;
        stack.push_back(Frame{rest, divisors_of(rest), 0});
    }
}

}  // namespace

at_status build_space(int tmpl, const int64_t* shape, int nshape, SpaceDesc& d,
                      std::vector<uint64_t>& factors) {
    std::memset(&d, 0, sizeof(d));
    factors.clear();
    // templates 2 and 3 are 0 and 1 with the vectorize and vthread knobs
    const bool annotated = tmpl == AT_TMPL_GEMM_VT || tmpl == AT_TMPL_CONV2D_NCHW_VT;
    if (annotated) tmpl -= 2;
    d.tmpl = tmpl;
    if (!shape || nshape < 1) return fail(AT_E_INVALID, "missing shape");
    for (int i = 0; i < nshape; ++i)
        if (shape[i] > 65535) return fail(AT_E_UNSUPPORTED, "shape value above 65535");
    std::vector<int64_t> extent;
    std::vector<int> levels;
    __int128 iters = 1;
    __int128 buf_size[N_BUFFERS] = {0, 0, 0};
    if (tmpl == AT_TMPL_GEMM) {
        if (nshape != 3) return fail(AT_E_INVALID, "GEMM shape must be {M, N, K}");
        int64_t M = shape[0], N = shape[1], K = shape[2];
        if (M < 1 || N < 1 || K < 1) return fail(AT_E_INVALID, "GEMM extents must be positive");
        // axes i, j, k; A[k][i], B[k][j], C[i][j]
        extent = {M, N, K};
        levels = {4, 4, 2};
        d.n_axes = 3;
        d.coef[0][2] = (int32_t)M; d.coef[0][0] = 1;     // A: k*M + i
        d.coef[1][2] = (int32_t)N; d.coef[1][1] = 1;     // B: k*N + j
        d.coef[2][0] = (int32_t)N; d.coef[2][1] = 1;     // C: i*N + j
        d.stride = 1;
        d.n_features = 10 * 11;
        iters = (__int128)M * N * K;
        buf_size[0] = (__int128)K * M; buf_size[1] = (__int128)K * N; buf_size[2] = (__int128)M * N;
    } else if (tmpl == AT_TMPL_CONV2D_NCHW) {
        if (nshape != 9) return fail(AT_E_INVALID, "conv2d shape must be {N,C,H,W,K,KH,KW,pad,stride}");
        int64_t Nb = shape[0], C = shape[1], H = shape[2], W = shape[3], K = shape[4];
        int64_t KH = shape[5], KW = shape[6], P = shape[7], S = shape[8];
        if (Nb != 1) return fail(AT_E_INVALID, "conv2d batch must be 1");
        if (C < 1 || H < 1 || W < 1 || K < 1 || KH < 1 || KW < 1 || P < 0 || S < 1)
            return fail(AT_E_INVALID, "conv2d sizes must be positive (pad >= 0)");
        int64_t Hp = H + 2 * P, Wp = W + 2 * P;
        if (Hp < KH || Wp < KW) return fail(AT_E_INVALID, "conv2d window larger than the padded input");
        int64_t OH = (Hp - KH) / S + 1, OW = (Wp - KW) / S + 1;
        // axes oc, oh, ow, rc, ry, rx
        extent = {K, OH, OW, C, KH, KW};
        levels = {4, 4, 4, 2, 2, 2};
        d.n_axes = 6;
        // data_pad[rc][oh*S + ry][ow*S + rx]
        d.coef[0][3] = (int32_t)(Hp * Wp); d.coef[0][1] = (int32_t)(S * Wp); d.coef[0][4] = (int32_t)Wp;
        d.coef[0][2] = (int32_t)S; d.coef[0][5] = 1;
        // kernel[oc][rc][ry][rx]
        d.coef[1][0] = (int32_t)(C * KH * KW); d.coef[1][3] = (int32_t)(KH * KW);
        d.coef[1][4] = (int32_t)KW; d.coef[1][5] = 1;
        // output[oc][oh][ow]
        d.coef[2][0] = (int32_t)(OH * OW); d.coef[2][1] = (int32_t)OW; d.coef[2][2] = 1;
        d.stride = (int32_t)S;
        d.n_features = 16 * 11;
        iters = (__int128)K * OH * OW * C * KH * KW;
        buf_size[0] = (__int128)C * Hp * Wp;
        buf_size[1] = (__int128)K * C * KH * KW;
        buf_size[2] = (__int128)K * OH * OW;
    } else {
        return fail(AT_E_INVALID, "unknown template");
    }
    const __int128 LIM = (__int128)1 << 31;
    for (int64_t e : extent)
        if (e > 65535) return fail(AT_E_UNSUPPORTED, "axis extent above 65535");
    if (tmpl == AT_TMPL_CONV2D_NCHW && (shape[2] + 2 * shape[7] > 65535 || shape[3] + 2 * shape[7] > 65535))
        return fail(AT_E_UNSUPPORTED, "padded input extent above 65535");
    if (iters >= LIM) return fail(AT_E_UNSUPPORTED, "loop nest has 2^31 or more iterations");
    for (int b = 0; b < N_BUFFERS; ++b)
        if (buf_size[b] >= LIM) return fail(AT_E_UNSUPPORTED, "buffer has 2^31 or more elements");

    int n_axes = d.n_axes;
    for (int a = 0; a < n_axes; ++a) {
        d.split_off[a] = (int32_t)factors.size();
        size_t before = factors.size();
        append_splits(extent[a], levels[a], factors);
        d.knob_size[a] = (uint32_t)(factors.size() - before);
    }
    d.knob_size[n_axes] = 3;       // auto_unroll_max_step in {0, 512, 1500}
    d.knob_size[n_axes + 1] = 2;   // unroll_explicit in {0, 1}
    d.n_knobs = n_axes + 2;
    if (annotated) {
        d.knob_size[n_axes + 2] = 2;   // vectorize in {0, 1}
        d.knob_size[n_axes + 3] = 2;   // vthread in {0, 1}
        d.n_knobs = n_axes + 4;
        d.ann_knobs = 1;
    }
    unsigned __int128 total = 1;
    for (int j = 0; j < d.n_knobs; ++j) total *= d.knob_size[j];
    if (total >= ((unsigned __int128)1 << 32))
        return fail(AT_E_UNSUPPORTED, "space holds 2^32 or more configurations");
    d.n_configs = (uint64_t)total;
    uint64_t r = 1;
    for (int j = d.n_knobs - 1; j >= 0; --j) {
        d.radix[j] = r;
        r *= d.knob_size[j];
    }
    d.n_mut = 0;
    for (int j = 0; j < d.n_knobs; ++j)
        if (d.knob_size[j] >= 2) d.mut[d.n_mut++] = j;
    return AT_OK;
}

}  // namespace at
