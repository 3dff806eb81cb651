// CPU ORACLE -- test infrastructure only.
//
// A plain, single-threaded, deliberately slow reference for the annealing hot
// path of "Learning to Optimize Tensor Programs" (Chen et al., NeurIPS 2018).
// Only the tests, the smoke check and the bench's CPU-baseline leg may load
// this library.  It shares no source with the HIP library: every step below
// (split enumeration, knob decoding, loop features, tree walk, Philox,
// thresholds, annealing, top-k) is written out again here, straight from the
// paper's definitions and the readings listed with each function.
//
// Build: g++ -O2 -std=c++17 -ffp-contract=off -fno-fast-math -shared -fPIC.
// All float arithmetic is single IEEE-754 operations (x86-64 SSE), so results
// are reproducible bit for bit.
//
// Pinning: every function here is checked by the CPU test-suite against
// something other than itself (hand-derived rows, brute-force enumeration of
// touched addresses, finite differences, closed-form counts, rocRAND's Philox,
// exhaustive search on small spaces, annealing invariants).

#include <cmath>
#include <cstdint>
#include <cstring>
#include <algorithm>
#include <string>
#include <vector>

namespace {

// ---------------------------------------------------------------------------
// Philox-4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As
// Easy as 1, 2, 3", SC 2011).  Round: two 32x32->64 multiplies with the
// published multipliers, Weyl key schedule with the published increments.
// ---------------------------------------------------------------------------
const uint32_t PHILOX_M0 = 0xD2511F53u;
const uint32_t PHILOX_M1 = 0xCD9E8D57u;
const uint32_t PHILOX_W0 = 0x9E3779B9u;
const uint32_t PHILOX_W1 = 0xBB67AE85u;

void philox4x32_10(const uint32_t key_in[2], const uint32_t ctr_in[4], uint32_t out[4]) {
    uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
    uint32_t k[2] = {key_in[0], key_in[1]};
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k[0] += PHILOX_W0;
            k[1] += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c[0];
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c[2];
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c[1] ^ k[0];
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c[3] ^ k[1];
        uint32_t n3 = lo0;
        c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    }
    for (int i = 0; i < 4; ++i) out[i] = c[i];
}

// Philox block for a 64-bit seed and four counter words.
void philox_block(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t out[4]) {
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t ctr[4] = {c0, c1, c2, c3};
    philox4x32_10(key, ctr, out);
}

// Uniform integer in [0, n) from one 32-bit word: floor(r * n / 2^32)
// (Lemire's multiply-shift range reduction, without rejection).
uint32_t range_reduce(uint32_t r, uint32_t n) {
    return (uint32_t)(((uint64_t)r * (uint64_t)n) >> 32);
}

// bitlen(x) = number of bits needed to write x: 0 for 0, floor(log2 x)+1 else.
int32_t bitlen(int64_t x) {
    int32_t b = 0;
    while (x > 0) { ++b; x >>= 1; }
    return b;
}

// ---------------------------------------------------------------------------
// Schedule templates (Section 2: multi-level tiling of every loop axis, loop
// ordering, thread binding and unrolling annotations).
// ---------------------------------------------------------------------------
// Templates 2 and 3 are 0 and 1 with two annotation knobs more (the
// vectorization annotation of Section 2's search space, and virtual-thread
// binding): vectorize in {0, 1} and vthread in {0, 1}, in that order after
// unroll_explicit.
enum { TMPL_GEMM = 0, TMPL_CONV2D = 1, TMPL_GEMM_VT = 2, TMPL_CONV2D_VT = 3 };

// Annotation ids of the loop-context "annotation" column (Appendix A.2).
// The one-hot form of the column has one column per id, ANN_KINDS in all
// (parallel is a CPU annotation that these GPU templates never produce).
enum {
    ANN_SERIAL = 0, ANN_UNROLL = 1, ANN_UNROLL_EXPLICIT = 2,
    ANN_BLOCK_X = 3, ANN_BLOCK_Y = 4, ANN_BLOCK_Z = 5,
    ANN_THREAD_X = 6, ANN_THREAD_Y = 7, ANN_THREAD_Z = 8,
    ANN_VTHREAD = 9, ANN_VECTORIZE = 10, ANN_PARALLEL = 11,
    ANN_KINDS = 12
};

// One term coef * axis inside one dimension of a buffer's index expression.
struct Term { int axis; int64_t coef; };
// One buffer dimension: its row-major element stride and its index terms.
struct Dim { int64_t stride; std::vector<Term> terms; };
struct Buffer { std::string name; std::vector<Dim> dims; };

// A loop of the generated nest: one level of one axis, or (fused kernel
// window loop) one level of two axes with the first one outer.
struct LoopComp { int axis; int level; };
struct Loop { std::vector<LoopComp> comps; int binding; };

// A tunable knob.  Split knobs choose an ordered factorization of an axis
// extent; value knobs choose one integer from a list.
struct Knob {
    bool is_split;
    int axis;                                  // split knobs
    std::vector<std::vector<int64_t>> splits;  // split knobs: factor tuples, outer level first
    std::vector<int64_t> values;               // value knobs
    int64_t size() const { return is_split ? (int64_t)splits.size() : (int64_t)values.size(); }
};

struct Space {
    int tmpl;
    std::vector<int64_t> shape;
    std::vector<int64_t> axis_extent;   // per axis
    std::vector<int> axis_levels;       // number of tiling levels per axis
    std::vector<Knob> knobs;
    int knob_auto_unroll;               // index of the auto_unroll_max_step knob
    int knob_unroll_explicit;           // index of the unroll_explicit knob
    int knob_vectorize = -1;            // index of the vectorize knob (templates 2, 3), else -1
    int knob_vthread = -1;              // index of the vthread knob (templates 2, 3), else -1
    std::vector<int> spatial_axes;      // axes whose third tiling level a vthread knob binds
    std::vector<int> axis_knob;         // split knob of each axis
    std::vector<Loop> loops;            // outer to inner
    std::vector<Buffer> buffers;
    uint64_t n_configs;
};

// All ordered k-factor splits of n, lexicographically ascending in
// (f_1, ..., f_k) with f_1 the outermost level.
void enumerate_splits(int64_t n, int k, std::vector<int64_t>& prefix,
                      std::vector<std::vector<int64_t>>& out) {
    if (k == 1) {
        prefix.push_back(n);
        out.push_back(prefix);
        prefix.pop_back();
        return;
    }
    for (int64_t f = 1; f <= n; ++f) {
        if (n % f != 0) continue;
        prefix.push_back(f);
        enumerate_splits(n / f, k - 1, prefix, out);
        prefix.pop_back();
    }
}

Knob split_knob(int axis, int64_t extent, int levels) {
    Knob kb;
    kb.is_split = true;
    kb.axis = axis;
    std::vector<int64_t> prefix;
    enumerate_splits(extent, levels, prefix, kb.splits);
    return kb;
}

Knob value_knob(std::vector<int64_t> values) {
    Knob kb;
    kb.is_split = false;
    kb.axis = -1;
    kb.values = values;
    return kb;
}

// GEMM C[i,j] = sum_k A[k,i] * B[k,j] (the running example of Section 2).
// A is [K][M], B is [K][N], C is [M][N], all row-major.
// Knobs: 4-level split of i, 4-level split of j, 2-level split of k,
// auto_unroll_max_step in {0, 512, 1500}, unroll_explicit in {0, 1}.
// Nest (outer to inner): i1 j1 i2 j2 k1 i3 j3 k2 i4 j4, with i1/j1 bound to
// blockIdx.y/x and i2/j2 to threadIdx.y/x.
bool build_gemm(Space& sp, const int64_t* shape, int nshape) {
    if (nshape != 3) return false;
    int64_t M = shape[0], N = shape[1], K = shape[2];
    if (M < 1 || N < 1 || K < 1) return false;
    enum { I = 0, J = 1, KK = 2 };
    sp.axis_extent = {M, N, K};
    sp.axis_levels = {4, 4, 2};
    sp.knobs.push_back(split_knob(I, M, 4));
    sp.knobs.push_back(split_knob(J, N, 4));
    sp.knobs.push_back(split_knob(KK, K, 2));
    sp.knobs.push_back(value_knob({0, 512, 1500}));
    sp.knobs.push_back(value_knob({0, 1}));
    sp.axis_knob = {0, 1, 2};
    sp.knob_auto_unroll = 3;
    sp.knob_unroll_explicit = 4;
    sp.spatial_axes = {I, J};
    auto L = [](int axis, int level, int binding) { Loop l; l.comps = {{axis, level}}; l.binding = binding; return l; };
    sp.loops = {L(I, 0, ANN_BLOCK_Y), L(J, 0, ANN_BLOCK_X), L(I, 1, ANN_THREAD_Y), L(J, 1, ANN_THREAD_X),
                L(KK, 0, ANN_SERIAL), L(I, 2, ANN_SERIAL), L(J, 2, ANN_SERIAL), L(KK, 1, ANN_SERIAL),
                L(I, 3, ANN_SERIAL), L(J, 3, ANN_SERIAL)};
    Buffer A{"A", {Dim{M, {{KK, 1}}}, Dim{1, {{I, 1}}}}};
    Buffer B{"B", {Dim{N, {{KK, 1}}}, Dim{1, {{J, 1}}}}};
    Buffer C{"C", {Dim{N, {{I, 1}}}, Dim{1, {{J, 1}}}}};
    sp.buffers = {A, B, C};
    return true;
}

// conv2d, NCHW, batch 1:
//   out[k][oh][ow] = sum_{c,ry,rx} data[c][oh*S+ry][ow*S+rx] * kernel[k][c][ry][rx]
// data is the zero-padded input [C][H+2p][W+2p]; coordinates are not clipped.
// Knobs: 4-level splits of oc, oh, ow; 2-level splits of rc, ry, rx;
// auto_unroll_max_step; unroll_explicit.
// Nest (16 loops): oc1 oh1 ow1 | oc2 oh2 ow2 | rc1 r1 | oc3 oh3 ow3 | rc2 r2 |
// oc4 oh4 ow4, where r_l fuses ry_l (outer) and rx_l of the same level.  The
// first band is bound to blockIdx.z/y/x and the second to threadIdx.z/y/x.
bool build_conv(Space& sp, const int64_t* shape, int nshape) {
    if (nshape != 9) return false;
    int64_t Nb = shape[0], C = shape[1], H = shape[2], W = shape[3], K = shape[4];
    int64_t KH = shape[5], KW = shape[6], P = shape[7], S = shape[8];
    if (Nb != 1 || C < 1 || H < 1 || W < 1 || K < 1 || KH < 1 || KW < 1 || P < 0 || S < 1) return false;
    int64_t Hp = H + 2 * P, Wp = W + 2 * P;
    if (Hp < KH || Wp < KW) return false;
    int64_t OH = (Hp - KH) / S + 1, OW = (Wp - KW) / S + 1;
    enum { OC = 0, OHX = 1, OWX = 2, RC = 3, RY = 4, RX = 5 };
    sp.axis_extent = {K, OH, OW, C, KH, KW};
    sp.axis_levels = {4, 4, 4, 2, 2, 2};
    sp.knobs.push_back(split_knob(OC, K, 4));
    sp.knobs.push_back(split_knob(OHX, OH, 4));
    sp.knobs.push_back(split_knob(OWX, OW, 4));
    sp.knobs.push_back(split_knob(RC, C, 2));
    sp.knobs.push_back(split_knob(RY, KH, 2));
    sp.knobs.push_back(split_knob(RX, KW, 2));
    sp.knobs.push_back(value_knob({0, 512, 1500}));
    sp.knobs.push_back(value_knob({0, 1}));
    sp.axis_knob = {0, 1, 2, 3, 4, 5};
    sp.knob_auto_unroll = 6;
    sp.knob_unroll_explicit = 7;
    sp.spatial_axes = {OC, OHX, OWX};
    auto L = [](int axis, int level, int binding) { Loop l; l.comps = {{axis, level}}; l.binding = binding; return l; };
    auto R = [](int level) { Loop l; l.comps = {{RY, level}, {RX, level}}; l.binding = ANN_SERIAL; return l; };
    sp.loops = {L(OC, 0, ANN_BLOCK_Z), L(OHX, 0, ANN_BLOCK_Y), L(OWX, 0, ANN_BLOCK_X),
                L(OC, 1, ANN_THREAD_Z), L(OHX, 1, ANN_THREAD_Y), L(OWX, 1, ANN_THREAD_X),
                L(RC, 0, ANN_SERIAL), R(0),
                L(OC, 2, ANN_SERIAL), L(OHX, 2, ANN_SERIAL), L(OWX, 2, ANN_SERIAL),
                L(RC, 1, ANN_SERIAL), R(1),
                L(OC, 3, ANN_SERIAL), L(OHX, 3, ANN_SERIAL), L(OWX, 3, ANN_SERIAL)};
    Buffer data{"data", {Dim{Hp * Wp, {{RC, 1}}}, Dim{Wp, {{OHX, S}, {RY, 1}}}, Dim{1, {{OWX, S}, {RX, 1}}}}};
    Buffer kern{"kernel", {Dim{C * KH * KW, {{OC, 1}}}, Dim{KH * KW, {{RC, 1}}}, Dim{KW, {{RY, 1}}}, Dim{1, {{RX, 1}}}}};
    Buffer out{"output", {Dim{OH * OW, {{OC, 1}}}, Dim{OW, {{OHX, 1}}}, Dim{1, {{OWX, 1}}}}};
    sp.buffers = {data, kern, out};
    return true;
}

// The annotation knobs of templates 2 and 3 (a reading of Section 2, whose
// search space takes unrolling and vectorization annotations): vectorize = 1 marks
// the innermost loop vectorized; vthread = 1 binds the third tiling level of
// every spatial axis (GEMM i3 j3, conv2d oc3 oh3 ow3) to virtual threads.
// Either annotation takes the place of the unroll rule on its loops; the
// nest and every other feature are unchanged.
void add_annotation_knobs(Space& sp) {
    sp.knob_vectorize = (int)sp.knobs.size();
    sp.knobs.push_back(value_knob({0, 1}));
    sp.knob_vthread = (int)sp.knobs.size();
    sp.knobs.push_back(value_knob({0, 1}));
}

// Knob values of configuration index cfg: mixed radix, knob 0 most significant.
void decode(const Space& sp, uint64_t cfg, std::vector<int64_t>& v) {
    int n = (int)sp.knobs.size();
    v.assign(n, 0);
    for (int j = n - 1; j >= 0; --j) {
        uint64_t sz = (uint64_t)sp.knobs[j].size();
        v[j] = (int64_t)(cfg % sz);
        cfg /= sz;
    }
}

uint64_t encode(const Space& sp, const std::vector<int64_t>& v) {
    uint64_t cfg = 0;
    for (size_t j = 0; j < sp.knobs.size(); ++j) cfg = cfg * (uint64_t)sp.knobs[j].size() + (uint64_t)v[j];
    return cfg;
}

// Per-loop raw quantities of one configuration (Appendix A.2 loop context).
struct LoopQ {
    int64_t ext, ann, bottom_up;
    std::vector<int64_t> touched, reuse, stride;  // per buffer
};

// Number of distinct values of s*x + y for x in a run of A consecutive
// integers and y in a run of B consecutive integers (s >= 1).  The windows
// [s*x, s*x+B) of consecutive x overlap or abut when B >= s, giving one run
// of (A-1)*s + B values; otherwise they are disjoint, giving A*B.
int64_t distinct_affine(int64_t A, int64_t B, int64_t s) {
    if (A == 1 || B >= s) return (A - 1) * s + B;
    return A * B;
}

void loop_quantities(const Space& sp, const std::vector<int64_t>& v, std::vector<LoopQ>& q) {
    int n_axes = (int)sp.axis_extent.size();
    // factor[a][l]: extent of level l of axis a under this configuration.
    std::vector<std::vector<int64_t>> factor(n_axes);
    for (int a = 0; a < n_axes; ++a) {
        const Knob& kb = sp.knobs[sp.axis_knob[a]];
        factor[a] = kb.splits[v[sp.axis_knob[a]]];
    }
    int64_t auto_unroll = sp.knobs[sp.knob_auto_unroll].values[v[sp.knob_auto_unroll]];
    int64_t explicit_unroll = sp.knobs[sp.knob_unroll_explicit].values[v[sp.knob_unroll_explicit]];
    const bool vectorize = sp.knob_vectorize >= 0 && sp.knobs[sp.knob_vectorize].values[v[sp.knob_vectorize]] == 1;
    const bool vthread = sp.knob_vthread >= 0 && sp.knobs[sp.knob_vthread].values[v[sp.knob_vthread]] == 1;

    int n_loops = (int)sp.loops.size();
    int n_buf = (int)sp.buffers.size();
    q.assign(n_loops, LoopQ{});
    for (int p = 0; p < n_loops; ++p) {
        const Loop& lp = sp.loops[p];
        LoopQ& o = q[p];
        // length
        o.ext = 1;
        for (const LoopComp& c : lp.comps) o.ext *= factor[c.axis][c.level];
        // bottom-up: product of the lengths of this loop and every loop inside it
        o.bottom_up = 1;
        for (int r = p; r < n_loops; ++r)
            for (const LoopComp& c : sp.loops[r].comps) o.bottom_up *= factor[c.axis][c.level];
        // range of each axis covered by the sub-nest rooted at this loop: the
        // product of that axis's levels found at or inside this loop
        std::vector<int64_t> range(n_axes, 1);
        for (int r = p; r < n_loops; ++r)
            for (const LoopComp& c : sp.loops[r].comps) range[c.axis] *= factor[c.axis][c.level];
        // annotation: thread binding, else unrolled when the whole sub-nest has
        // at most auto_unroll_max_step iterations, else serial
        bool third_spatial = false;
        for (int a : sp.spatial_axes)
            if (lp.comps.size() == 1 && lp.comps[0].axis == a && lp.comps[0].level == 2) third_spatial = true;
        if (lp.binding != ANN_SERIAL) o.ann = lp.binding;
        else if (vthread && third_spatial) o.ann = ANN_VTHREAD;
        else if (vectorize && p == n_loops - 1) o.ann = ANN_VECTORIZE;
        else if (auto_unroll > 0 && o.bottom_up <= auto_unroll) o.ann = explicit_unroll ? ANN_UNROLL_EXPLICIT : ANN_UNROLL;
        else o.ann = ANN_SERIAL;

        o.touched.assign(n_buf, 0);
        o.reuse.assign(n_buf, 0);
        o.stride.assign(n_buf, 0);
        for (int b = 0; b < n_buf; ++b) {
            const Buffer& buf = sp.buffers[b];
            // touch count: distinct elements = product over dimensions of the
            // distinct index values of that dimension
            int64_t touched = 1;
            for (const Dim& d : buf.dims) {
                if (d.terms.size() == 1) {
                    touched *= range[d.terms[0].axis];
                } else {
                    // s*x + y with x the output axis (coef s) and y the window axis (coef 1)
                    const Term& tx = d.terms[0];
                    const Term& ty = d.terms[1];
                    touched *= distinct_affine(range[tx.axis], range[ty.axis], tx.coef);
                }
            }
            o.touched[b] = touched;
            o.reuse[b] = o.bottom_up / touched;
            // stride: coefficient of this loop's variable in the buffer's
            // flattened index.  A level-l variable of axis a enters a with weight
            // prod(factors of a below level l); a enters the flat index with
            // sum over dims of dim.stride * term.coef.
            auto coef_of_axis = [&](int axis) {
                int64_t c = 0;
                for (const Dim& d : buf.dims)
                    for (const Term& t : d.terms)
                        if (t.axis == axis) c += d.stride * t.coef;
                return c;
            };
            auto var_coef = [&](const LoopComp& c) {
                int64_t inner = 1;
                for (int l = c.level + 1; l < sp.axis_levels[c.axis]; ++l) inner *= factor[c.axis][l];
                return coef_of_axis(c.axis) * inner;
            };
            if (lp.comps.size() == 1) {
                o.stride[b] = var_coef(lp.comps[0]);
            } else {
                // fused window loop r with ry = r div RX, rx = r mod RX: the
                // flat index changes, for one step of r from its first
                // iteration, by rx's weight when RX > 1 and by ry's otherwise
                const LoopComp& cy = lp.comps[0];
                const LoopComp& cx = lp.comps[1];
                int64_t ext_x = factor[cx.axis][cx.level];
                o.stride[b] = (ext_x > 1) ? var_coef(cx) : var_coef(cy);
            }
        }
    }
}

// Feature row: per loop, outer to inner: bitlen(length), annotation id, then
// for each buffer bitlen(touch count), bitlen(reuse ratio), bitlen(stride).
void features_of(const Space& sp, uint64_t cfg, int32_t* row) {
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    std::vector<LoopQ> q;
    loop_quantities(sp, v, q);
    int k = 0;
    for (const LoopQ& o : q) {
        row[k++] = bitlen(o.ext);
        row[k++] = (int32_t)o.ann;
        for (size_t b = 0; b < o.touched.size(); ++b) {
            row[k++] = bitlen(o.touched[b]);
            row[k++] = bitlen(o.reuse[b]);
            row[k++] = bitlen(o.stride[b]);
        }
    }
}

int n_features_of(const Space& sp) { return (int)sp.loops.size() * (2 + 3 * (int)sp.buffers.size()); }

// Feature row with the top-down and bottom-up columns of Appendix A.2: per
// loop, outer to inner: bitlen(length), annotation id, bitlen(top-down),
// bitlen(bottom-up), then for each buffer bitlen(touch count), bitlen(reuse
// ratio), bitlen(stride).  Top-down is the product of the lengths of the
// loops strictly outside the loop (1 for the outermost), bottom-up that of
// the loop and the loops inside it.
void features_full_of(const Space& sp, uint64_t cfg, int32_t* row) {
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    std::vector<LoopQ> q;
    loop_quantities(sp, v, q);
    int64_t top_down = 1;
    int k = 0;
    for (const LoopQ& o : q) {
        row[k++] = bitlen(o.ext);
        row[k++] = (int32_t)o.ann;
        row[k++] = bitlen(top_down);
        row[k++] = bitlen(o.bottom_up);
        for (size_t b = 0; b < o.touched.size(); ++b) {
            row[k++] = bitlen(o.touched[b]);
            row[k++] = bitlen(o.reuse[b]);
            row[k++] = bitlen(o.stride[b]);
        }
        top_down *= o.ext;
    }
}

int n_features_full_of(const Space& sp) { return (int)sp.loops.size() * (4 + 3 * (int)sp.buffers.size()); }

// The loop-context table of Appendix A.2 with its annotation column in
// one-hot form: per loop, outer to inner: bitlen(length), ANN_KINDS columns
// holding 1 for the loop's annotation and 0 for every other, bitlen(top-down),
// bitlen(bottom-up), then for each buffer bitlen(touch count), bitlen(reuse
// ratio), bitlen(stride).
void features_onehot_of(const Space& sp, uint64_t cfg, int32_t* row) {
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    std::vector<LoopQ> q;
    loop_quantities(sp, v, q);
    int64_t top_down = 1;
    int k = 0;
    for (const LoopQ& o : q) {
        row[k++] = bitlen(o.ext);
        for (int a = 0; a < ANN_KINDS; ++a) row[k++] = (o.ann == a) ? 1 : 0;
        row[k++] = bitlen(top_down);
        row[k++] = bitlen(o.bottom_up);
        for (size_t b = 0; b < o.touched.size(); ++b) {
            row[k++] = bitlen(o.touched[b]);
            row[k++] = bitlen(o.reuse[b]);
            row[k++] = bitlen(o.stride[b]);
        }
        top_down *= o.ext;
    }
}

int n_features_onehot_of(const Space& sp) {
    return (int)sp.loops.size() * (3 + ANN_KINDS + 3 * (int)sp.buffers.size());
}

// ---------------------------------------------------------------------------
// Context relation features (Section 4; Appendix A.2 "Relation Feature").
// Over the loops of the nest's longest chain (here the whole perfect nest),
// with Z_ki the i-th context feature of loop k and log2-spaced thresholds
// beta_t, R_t^(ij) = max over the loops k with Z_kj < beta_t of Z_ki.  The
// two pairs of the appendix, per buffer b: reuse ratio against touch count,
// and top-down against touch count.
// Readings: beta_t = 2^t for t = 1..32; the maximised value is taken in the
// same bitlen space as the loop features (bitlen of the reuse ratio, bitlen
// of the top-down product); top-down is the product of the lengths of the
// loops strictly outside loop k (1 for the outermost); a threshold that no
// loop meets gives 0.  Row layout: [pair][buffer][t - 1], pair 0 the reuse
// relation, pair 1 the top-down one.
// ---------------------------------------------------------------------------
const int REL_THRESHOLDS = 32;

int n_relation_features_of(const Space& sp) { return 2 * (int)sp.buffers.size() * REL_THRESHOLDS; }

void relation_features_of(const Space& sp, uint64_t cfg, int32_t* row) {
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    std::vector<LoopQ> q;
    loop_quantities(sp, v, q);
    const int n_loops = (int)q.size(), n_buf = (int)sp.buffers.size();
    std::vector<int64_t> top_down(n_loops, 1);
    for (int k = 1; k < n_loops; ++k) top_down[k] = top_down[k - 1] * q[k - 1].ext;
    for (int b = 0; b < n_buf; ++b) {
        for (int t = 1; t <= REL_THRESHOLDS; ++t) {
            const int64_t beta = (int64_t)1 << t;
            int32_t r_reuse = 0, r_top = 0;
            for (int k = 0; k < n_loops; ++k) {
                if (q[k].touched[b] < beta) {
                    r_reuse = std::max(r_reuse, bitlen(q[k].reuse[b]));
                    r_top = std::max(r_top, bitlen(top_down[k]));
                }
            }
            row[(0 * n_buf + b) * REL_THRESHOLDS + (t - 1)] = r_reuse;
            row[(1 * n_buf + b) * REL_THRESHOLDS + (t - 1)] = r_top;
        }
    }
}

// ---------------------------------------------------------------------------
// Gradient-boosted tree ensemble (Section 3.1).  Full depth-d trees in heap
// order: node n has children 2n+1 (taken when x[fid] < thr) and 2n+2.  The
// prediction is the fp32 sum of the reached leaves, added one tree after the
// other in tree order starting from +0.0f.
// ---------------------------------------------------------------------------
struct Ensemble {
    int n_trees, depth, n_features;
    const uint8_t* fid;   // [T][2^d - 1]
    const uint8_t* thr;   // [T][2^d - 1]
    const float* leaf;    // [T][2^d]
};

int leaf_index(const Ensemble& e, int t, const int32_t* x) {
    int64_t n_int = ((int64_t)1 << e.depth) - 1;
    const uint8_t* f = e.fid + (int64_t)t * n_int;
    const uint8_t* th = e.thr + (int64_t)t * n_int;
    int64_t n = 0;
    for (int l = 0; l < e.depth; ++l) {
        if (x[f[n]] < (int32_t)th[n]) n = 2 * n + 1;
        else n = 2 * n + 2;
    }
    return (int)(n - n_int);
}

float predict_row(const Ensemble& e, const int32_t* x, uint16_t* leaves) {
    float s = 0.0f;
    int64_t n_leaf = (int64_t)1 << e.depth;
    for (int t = 0; t < e.n_trees; ++t) {
        int li = leaf_index(e, t, x);
        if (leaves) leaves[t] = (uint16_t)li;
        s = s + e.leaf[(int64_t)t * n_leaf + li];
    }
    return s;
}

// ---------------------------------------------------------------------------
// Parallel simulated annealing with the model score as negative energy
// (Section 3.3, Algorithm 1).  Counter-based randomness keyed by the global
// chain id keeps every chain independent of the others.
// ---------------------------------------------------------------------------
struct TopEntry { uint64_t cfg; float score; uint32_t valid; };

// Entries precede each other by higher score, then by lower config index.
bool precedes(float sa, uint64_t ca, float sb, uint64_t cb) {
    if (sa > sb) return true;
    if (sa < sb) return false;
    return ca < cb;
}

// Offer a scored configuration to a chain's top-k list (count entries valid).
void topk_offer(TopEntry* list, int k, uint64_t cfg, float score) {
    int count = 0;
    while (count < k && list[count].valid) ++count;
    for (int i = 0; i < count; ++i)
        if (list[i].cfg == cfg) return;
    if (count == k && !precedes(score, cfg, list[k - 1].score, list[k - 1].cfg)) return;
    // insertion position: after every entry that precedes the new one
    int pos = 0;
    while (pos < count && precedes(list[pos].score, list[pos].cfg, score, cfg)) ++pos;
    int last = (count < k) ? count : k - 1;
    for (int i = last; i > pos; --i) list[i] = list[i - 1];
    list[pos] = TopEntry{cfg, score, 1u};
}

// Metropolis threshold for step s of a call of `steps` steps: accept a move
// with score change delta with probability min(1, exp(delta / T_s)), i.e. iff
// u <= exp(delta/T) <=> T*ln(u) <= delta.  T_s falls linearly from 1 to 0.
float threshold(uint64_t seed, uint64_t chain, uint64_t step_abs, int s, int steps) {
    uint32_t r[4];
    philox_block(seed, (uint32_t)chain, (uint32_t)step_abs, 0u, 0u, r);
    double T = (steps == 1) ? 0.0 : 1.0 - (double)s / (double)(steps - 1);
    double u = ((double)r[2] + 0.5) * (1.0 / 4294967296.0);
    return (float)(T * std::log(u));
}

float score_config(const Space& sp, const Ensemble& e, uint64_t cfg) {
    std::vector<int32_t> row(n_features_of(sp));
    features_of(sp, cfg, row.data());
    return predict_row(e, row.data(), nullptr);
}

// Eq. 4 (Section 4): f_hat = f_hat_global + f_hat_local.  The global model
// reads the invariant representation (the context relation features), the
// in-domain local model the loop-context features; each prediction is its
// own fp32 fold in tree order, and the two are added once, global first.
float score_config_global_local(const Space& sp, const Ensemble& global, const Ensemble& local, uint64_t cfg) {
    std::vector<int32_t> rel(n_relation_features_of(sp));
    relation_features_of(sp, cfg, rel.data());
    const float g = predict_row(global, rel.data(), nullptr);
    std::vector<int32_t> row(n_features_of(sp));
    features_of(sp, cfg, row.data());
    const float l = predict_row(local, row.data(), nullptr);
    return g + l;
}

// ---------------------------------------------------------------------------
// Picking the batch to measure (Algorithm 1 after the annealing; Section 3.3,
// Eq. 3).  Q is the set of distinct configurations the chains keep.  From
// the top `pool` of Q (the paper's top lambda*b, ordered by score, higher
// first, then by index) a greedy submodular maximisation of
//     L(S) = sum_{s in S} score(s) + alpha * sum_j |{ s_j : s in S }|
// (Eq. 3 with score = -f_hat) picks n_greedy configurations one at a time:
// each pick maximises the marginal gain L(S + {s}) - L(S), which is score(s)
// plus alpha times the number of knobs j whose value s_j no pick in S has.
// Readings: the gain is evaluated in fp32 as score + alpha * count (one
// product, one sum); ties go to the earlier configuration in pool order.
// Then epsilon-greedy: n_random configurations drawn uniformly among those of
// S_e not yet selected; draw i uses Philox block (i, 0, 5, 0) under `seed`,
// u = r1 * 2^32 + r0, and takes the floor(u * remaining / 2^64)-th
// unselected configuration in index order.
// ---------------------------------------------------------------------------
// Writes n_greedy + n_random entries: greedy picks (flag 1) in pick order,
// then random picks (flag 2, score 0); slots left empty have flag 0.
void select_batch(const Space& sp, const TopEntry* cand, int64_t n_cand, int pool, int n_greedy, float alpha,
                  int n_random, uint64_t seed, TopEntry* out) {
    // Q: distinct valid configurations
    std::vector<TopEntry> q;
    for (int64_t i = 0; i < n_cand; ++i)
        if (cand[i].valid) q.push_back(TopEntry{cand[i].cfg, cand[i].score, 1u});
    std::sort(q.begin(), q.end(),
              [](const TopEntry& a, const TopEntry& b) { return precedes(a.score, a.cfg, b.score, b.cfg); });
    std::vector<TopEntry> distinct;
    for (const TopEntry& e : q)
        if (distinct.empty() || distinct.back().cfg != e.cfg) distinct.push_back(e);
    // the top `pool` of Q
    if ((int64_t)distinct.size() > pool) distinct.resize(pool);
    const int m = (int)sp.knobs.size();
    std::vector<std::vector<int64_t>> vals(distinct.size());
    for (size_t i = 0; i < distinct.size(); ++i) decode(sp, distinct[i].cfg, vals[i]);
    // greedy maximisation of L
    std::vector<std::vector<int64_t>> covered(m);   // knob values already in S
    std::vector<bool> taken(distinct.size(), false);
    for (int i = 0; i < n_greedy + n_random; ++i) out[i] = TopEntry{0, 0.0f, 0u};
    std::vector<uint64_t> selected;
    int picks = 0;
    for (int step = 0; step < n_greedy && step < (int)distinct.size(); ++step) {
        int best = -1;
        float best_gain = 0.0f;
        for (size_t i = 0; i < distinct.size(); ++i) {
            if (taken[i]) continue;
            int fresh = 0;
            for (int j = 0; j < m; ++j)
                if (std::find(covered[j].begin(), covered[j].end(), vals[i][j]) == covered[j].end()) ++fresh;
            float cov = alpha * (float)fresh;
            float gain = distinct[i].score + cov;
            if (best < 0 || gain > best_gain) {
                best = (int)i;
                best_gain = gain;
            }
        }
        taken[best] = true;
        for (int j = 0; j < m; ++j)
            if (std::find(covered[j].begin(), covered[j].end(), vals[best][j]) == covered[j].end())
                covered[j].push_back(vals[best][j]);
        out[picks++] = TopEntry{distinct[best].cfg, distinct[best].score, 1u};
        selected.push_back(distinct[best].cfg);
    }
    // epsilon-greedy: uniform over the configurations not selected yet
    for (int i = 0; i < n_random; ++i) {
        std::sort(selected.begin(), selected.end());
        uint64_t remaining = sp.n_configs - (uint64_t)selected.size();
        if (remaining == 0) break;
        uint32_t r[4];
        philox_block(seed, (uint32_t)i, 0u, 5u, 0u, r);
        unsigned __int128 u = ((unsigned __int128)r[1] << 32) | r[0];
        uint64_t k = (uint64_t)((u * remaining) >> 64);
        // the k-th configuration (0-based, ascending) that is not selected
        uint64_t cfg = k;
        for (uint64_t x : selected) {
            if (x <= cfg) ++cfg;
            else break;
        }
        out[picks++] = TopEntry{cfg, 0.0f, 2u};
        selected.push_back(cfg);
    }
}

}  // namespace

// ===========================================================================
// C API used by the tests (via ctypes).  Status: 0 ok, negative on error.
// ===========================================================================
extern "C" {

int or_space_create(int tmpl, const int64_t* shape, int nshape, void** out) {
    if (!out || !shape) return -1;
    Space* sp = new Space();
    sp->tmpl = tmpl;
    sp->shape.assign(shape, shape + nshape);
    bool ok = (tmpl == TMPL_GEMM || tmpl == TMPL_GEMM_VT) ? build_gemm(*sp, shape, nshape)
            : (tmpl == TMPL_CONV2D || tmpl == TMPL_CONV2D_VT) ? build_conv(*sp, shape, nshape) : false;
    if (!ok) { delete sp; return -1; }
    if (tmpl == TMPL_GEMM_VT || tmpl == TMPL_CONV2D_VT) add_annotation_knobs(*sp);
    sp->n_configs = 1;
    for (const Knob& kb : sp->knobs) sp->n_configs *= (uint64_t)kb.size();
    *out = sp;
    return 0;
}

void or_space_destroy(void* h) { delete (Space*)h; }

int or_space_info(void* h, int* n_knobs, int64_t* knob_sizes, int* n_loops, int* n_features, uint64_t* n_configs) {
    const Space& sp = *(Space*)h;
    if (n_knobs) *n_knobs = (int)sp.knobs.size();
    if (knob_sizes) for (size_t j = 0; j < sp.knobs.size(); ++j) knob_sizes[j] = sp.knobs[j].size();
    if (n_loops) *n_loops = (int)sp.loops.size();
    if (n_features) *n_features = n_features_of(sp);
    if (n_configs) *n_configs = sp.n_configs;
    return 0;
}

// Factors of value `idx` of split knob `knob` (outer level first); returns the level count.
int or_knob_split(void* h, int knob, int64_t idx, int64_t* factors) {
    const Space& sp = *(Space*)h;
    if (knob < 0 || knob >= (int)sp.knobs.size() || !sp.knobs[knob].is_split) return -1;
    if (idx < 0 || idx >= sp.knobs[knob].size()) return -1;
    const std::vector<int64_t>& f = sp.knobs[knob].splits[idx];
    for (size_t l = 0; l < f.size(); ++l) factors[l] = f[l];
    return (int)f.size();
}

int or_decode(void* h, uint64_t cfg, int64_t* values) {
    const Space& sp = *(Space*)h;
    if (cfg >= sp.n_configs) return -5;
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    for (size_t j = 0; j < v.size(); ++j) values[j] = v[j];
    return 0;
}

int or_encode(void* h, const int64_t* values, uint64_t* cfg) {
    const Space& sp = *(Space*)h;
    std::vector<int64_t> v(values, values + sp.knobs.size());
    for (size_t j = 0; j < v.size(); ++j)
        if (v[j] < 0 || v[j] >= sp.knobs[j].size()) return -5;
    *cfg = encode(sp, v);
    return 0;
}

// Raw per-loop quantities: for each loop, [ext, ann, bottom_up, then per
// buffer touched, reuse, stride] (int64).
int or_loop_quantities(void* h, uint64_t cfg, int64_t* out) {
    const Space& sp = *(Space*)h;
    if (cfg >= sp.n_configs) return -5;
    std::vector<int64_t> v;
    decode(sp, cfg, v);
    std::vector<LoopQ> q;
    loop_quantities(sp, v, q);
    int k = 0;
    for (const LoopQ& o : q) {
        out[k++] = o.ext;
        out[k++] = o.ann;
        out[k++] = o.bottom_up;
        for (size_t b = 0; b < o.touched.size(); ++b) {
            out[k++] = o.touched[b];
            out[k++] = o.reuse[b];
            out[k++] = o.stride[b];
        }
    }
    return 0;
}

int or_features(void* h, const uint64_t* cfgs, int64_t n, int32_t* feats) {
    const Space& sp = *(Space*)h;
    int F = n_features_of(sp);
    for (int64_t i = 0; i < n; ++i) {
        if (cfgs[i] >= sp.n_configs) return -5;
        features_of(sp, cfgs[i], feats + i * F);
    }
    return 0;
}

int or_features_onehot(void* h, const uint64_t* cfgs, int64_t n, int32_t* feats) {
    const Space& sp = *(Space*)h;
    int F = n_features_onehot_of(sp);
    for (int64_t i = 0; i < n; ++i) {
        if (cfgs[i] >= sp.n_configs) return -5;
        features_onehot_of(sp, cfgs[i], feats + i * F);
    }
    return 0;
}

int or_features_full(void* h, const uint64_t* cfgs, int64_t n, int32_t* feats) {
    const Space& sp = *(Space*)h;
    int F = n_features_full_of(sp);
    for (int64_t i = 0; i < n; ++i) {
        if (cfgs[i] >= sp.n_configs) return -5;
        features_full_of(sp, cfgs[i], feats + i * F);
    }
    return 0;
}

int or_predict(int n_trees, int depth, int n_features, const uint8_t* fid, const uint8_t* thr,
               const float* leaf, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves) {
    if (n_trees < 1 || depth < 1 || depth > 15 || n_features < 1) return -1;
    Ensemble e{n_trees, depth, n_features, fid, thr, leaf};
    int64_t n_int = ((int64_t)1 << depth) - 1;
    for (int64_t t = 0; t < (int64_t)n_trees * n_int; ++t)
        if (fid[t] >= n_features) return -1;
    for (int64_t i = 0; i < n; ++i)
        scores[i] = predict_row(e, feats + i * n_features, leaves ? leaves + i * n_trees : nullptr);
    return 0;
}

// Trees in node-list form, as a trained gradient-boosting library writes
// them out (Section 3.1: the model is such an ensemble; its trees need not be
// full nor share one depth).  Tree t owns nodes offsets[t] .. offsets[t+1]-1,
// its root first; child indices count from the tree's first node.  A node
// with left >= 0 is a split: the walk takes left when x[feature] <
// threshold, the two compared as doubles, else right.  A node with left < 0
// is a leaf worth value.  A row's score is the fp32 sum of its reached
// leaves, added in tree order from +0.0f, exactly as predict_row.  Returns -1
// for a child or feature out of range or a walk longer than its tree.
int or_predict_nodes(int n_trees, const int32_t* offsets, const int32_t* left, const int32_t* right,
                     const int32_t* feature, const float* threshold, const float* value, int n_features,
                     const int32_t* feats, int64_t n, float* scores) {
    if (n_trees < 1 || n_features < 1) return -1;
    for (int64_t i = 0; i < n; ++i) {
        const int32_t* x = feats + i * n_features;
        float s = 0.0f;
        for (int t = 0; t < n_trees; ++t) {
            const int32_t base = offsets[t], size = offsets[t + 1] - offsets[t];
            if (size < 1) return -1;
            int32_t node = 0;
            for (int32_t steps = 0; left[base + node] >= 0; ++steps) {
                if (steps >= size) return -1;
                const int32_t j = base + node;
                if (feature[j] < 0 || feature[j] >= n_features) return -1;
                node = (double)x[feature[j]] < (double)threshold[j] ? left[j] : right[j];
                if (node < 0 || node >= size) return -1;
            }
            s = s + value[base + node];
        }
        scores[i] = s;
    }
    return 0;
}

void or_philox(uint64_t seed, const uint32_t* ctr, uint32_t* out) {
    philox_block(seed, ctr[0], ctr[1], ctr[2], ctr[3], out);
}

int or_thresholds(uint64_t seed, int64_t chain0, int64_t n_chains, uint64_t step_base, int steps, float* thr) {
    if (steps < 1 || n_chains < 0) return -1;
    for (int64_t c = 0; c < n_chains; ++c)
        for (int s = 0; s < steps; ++s)
            thr[c * steps + s] = threshold(seed, (uint64_t)(chain0 + c), step_base + (uint64_t)s, s, steps);
    return 0;
}

// Annealing over a set of spaces sharing one ensemble.  Chain c (local index)
// belongs to space w with offsets[w] <= c < offsets[w+1]; its global id is
// chain0 + c.  Per-chain state (in/out): cur knob values [n][max_knobs],
// cur score, initialised flag, step_abs, top-k [n][k].  thr is [n][steps].
// trace (optional) receives [n][steps] entries (cfg, score, accepted).
}  // extern "C"

namespace {

// The annealing loop of or_sa_run; `global` set: the energy is Eq. 4's
// global + local model (score_config_global_local), else the ensemble e
// alone.
int sa_run(void** spaces, int n_spaces, const int64_t* offsets, const Ensemble& e, const Ensemble* global,
           uint64_t seed, int64_t chain0, int64_t n_chains, int topk, int steps, const float* thr, int max_knobs,
           int64_t* cur_knobs, float* cur_score, uint8_t* initialised, uint64_t* step_abs, TopEntry* tops,
           TopEntry* trace) {
    if (n_spaces < 1 || topk < 1 || steps < 0) return -1;
    if (offsets[0] != 0 || offsets[n_spaces] != n_chains) return -1;
    for (int64_t c = 0; c < n_chains; ++c) {
        int w = 0;
        while (!(offsets[w] <= c && c < offsets[w + 1])) ++w;
        const Space& sp = *(Space*)spaces[w];
        if (n_features_of(sp) != e.n_features) return -6;
        if (global && n_relation_features_of(sp) != global->n_features) return -6;
        auto score = [&](uint64_t cfg) {
            return global ? score_config_global_local(sp, *global, e, cfg) : score_config(sp, e, cfg);
        };
        int nk = (int)sp.knobs.size();
        if (nk > max_knobs) return -1;
        uint64_t g = (uint64_t)(chain0 + c);
        int64_t* v = cur_knobs + c * max_knobs;
        TopEntry* list = tops + c * topk;
        std::vector<int64_t> cur(v, v + nk);
        if (!initialised[c]) {
            // initial state: each knob value uniform over its range
            uint32_t r[4] = {0, 0, 0, 0};
            for (int j = 0; j < nk; ++j) {
                if (j % 4 == 0) philox_block(seed, (uint32_t)g, 0u, 1u, (uint32_t)(j / 4), r);
                cur[j] = range_reduce(r[j % 4], (uint32_t)sp.knobs[j].size());
            }
            for (int i = 0; i < topk; ++i) list[i] = TopEntry{0, 0.0f, 0u};
            uint64_t cfg0 = encode(sp, cur);
            cur_score[c] = score(cfg0);
            topk_offer(list, topk, cfg0, cur_score[c]);
            step_abs[c] = 0;
            initialised[c] = 1;
        }
        // the knobs a mutation can change: those with at least two values
        std::vector<int> mutable_knobs;
        for (int j = 0; j < nk; ++j)
            if (sp.knobs[j].size() >= 2) mutable_knobs.push_back(j);
        for (int s = 0; s < steps; ++s) {
            uint32_t r[4];
            philox_block(seed, (uint32_t)g, (uint32_t)step_abs[c], 0u, 0u, r);
            std::vector<int64_t> cand = cur;
            if (!mutable_knobs.empty()) {
                int j = mutable_knobs[range_reduce(r[0], (uint32_t)mutable_knobs.size())];
                int64_t nv = range_reduce(r[1], (uint32_t)(sp.knobs[j].size() - 1));
                if (nv >= cur[j]) nv += 1;   // uniform over the other values
                cand[j] = nv;
            }
            uint64_t cfg = encode(sp, cand);
            float sc = score(cfg);
            topk_offer(list, topk, cfg, sc);
            float delta = sc - cur_score[c];
            bool accept = delta >= thr[c * steps + s];
            if (accept) {
                cur = cand;
                cur_score[c] = sc;
            }
            if (trace) trace[c * steps + s] = TopEntry{cfg, sc, accept ? 1u : 0u};
            step_abs[c] += 1;
        }
        for (int j = 0; j < nk; ++j) v[j] = cur[j];
    }
    return 0;
}

}  // namespace

extern "C" {

// Annealing over a set of spaces sharing one ensemble.  Chain c (local index)
// belongs to space w with offsets[w] <= c < offsets[w+1]; its global id is
// chain0 + c.  Per-chain state (in/out): cur knob values [n][max_knobs],
// cur score, initialised flag, step_abs, top-k [n][k].  thr is [n][steps].
// trace (optional) receives [n][steps] entries (cfg, score, accepted).
int or_sa_run(void** spaces, int n_spaces, const int64_t* offsets,
              int n_trees, int depth, int n_features, const uint8_t* fid, const uint8_t* thr_nodes,
              const float* leaf, uint64_t seed, int64_t chain0, int64_t n_chains, int topk,
              int steps, const float* thr, int max_knobs,
              int64_t* cur_knobs, float* cur_score, uint8_t* initialised, uint64_t* step_abs,
              TopEntry* tops, TopEntry* trace) {
    const Ensemble e{n_trees, depth, n_features, fid, thr_nodes, leaf};
    return sa_run(spaces, n_spaces, offsets, e, nullptr, seed, chain0, n_chains, topk, steps, thr, max_knobs,
                  cur_knobs, cur_score, initialised, step_abs, tops, trace);
}

// or_sa_run whose energy is Eq. 4's sum of a global model over the context
// relation features (g_* arrays, g_n_features = 2 * buffers * 32) and the
// local model over the loop-context features (the usual ensemble arrays).
int or_sa_run_global_local(void** spaces, int n_spaces, const int64_t* offsets,
                           int g_n_trees, int g_depth, int g_n_features, const uint8_t* g_fid,
                           const uint8_t* g_thr, const float* g_leaf,
                           int n_trees, int depth, int n_features, const uint8_t* fid, const uint8_t* thr_nodes,
                           const float* leaf, uint64_t seed, int64_t chain0, int64_t n_chains, int topk,
                           int steps, const float* thr, int max_knobs,
                           int64_t* cur_knobs, float* cur_score, uint8_t* initialised, uint64_t* step_abs,
                           TopEntry* tops, TopEntry* trace) {
    const Ensemble e{n_trees, depth, n_features, fid, thr_nodes, leaf};
    const Ensemble g{g_n_trees, g_depth, g_n_features, g_fid, g_thr, g_leaf};
    return sa_run(spaces, n_spaces, offsets, e, &g, seed, chain0, n_chains, topk, steps, thr, max_knobs,
                  cur_knobs, cur_score, initialised, step_abs, tops, trace);
}

int or_relation_features(void* h, const uint64_t* cfgs, int64_t n, int32_t* feats) {
    const Space& sp = *(Space*)h;
    int F = n_relation_features_of(sp);
    for (int64_t i = 0; i < n; ++i) {
        if (cfgs[i] >= sp.n_configs) return -5;
        relation_features_of(sp, cfgs[i], feats + i * F);
    }
    return 0;
}

// Batch selection (see select_batch): cand [n_cand] entries, out
// [n_greedy + n_random] entries.
int or_select_batch(void* h, const TopEntry* cand, int64_t n_cand, int pool, int n_greedy, float alpha,
                    int n_random, uint64_t seed, TopEntry* out) {
    if (!h || n_cand < 0 || pool < 0 || n_greedy < 0 || n_random < 0) return -1;
    select_batch(*(Space*)h, cand, n_cand, pool, n_greedy, alpha, n_random, seed, out);
    return 0;
}

}  // extern "C"
