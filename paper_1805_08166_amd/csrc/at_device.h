// Device helpers shared by the HIP kernels: loop-context feature evaluation
// of the two schedule templates, the tree walk over LDS-resident node words,
// and best-list insertion.
#pragma once

#include "at_internal.h"

namespace at {
namespace dev {

constexpr int WG = 256;   // workgroup size of every kernel (4 wave64s)

// bitlen(x): bits needed to write x (0 for 0).
__device__ __forceinline__ uint32_t bitlen(uint32_t x) { return 32u - (uint32_t)__clz((int)x); }

// bitlen(floor(a / b)) for a >= b >= 1 without a division: with
// k = bitlen(a) - bitlen(b) >= 0 the quotient lies in [2^(k-1), 2^(k+1)),
// and it reaches 2^k exactly when floor(a / 2^k) >= b.
__device__ __forceinline__ uint32_t bitlen_quot(uint32_t a, uint32_t b) {
    uint32_t k = bitlen(a) - bitlen(b);
    return k + ((a >> k) >= b ? 1u : 0u);
}

// Distinct values of S*x + y for x over A consecutive integers and y over B
// consecutive integers: one run of (A-1)*S + B when the windows touch
// (B >= S, or a single x), else A*B isolated windows.
__device__ __forceinline__ uint32_t distinct_affine(uint32_t A, uint32_t B, uint32_t S) {
    return (A == 1u || B >= S) ? (A - 1u) * S + B : A * B;
}

// --------------------------------------------------------------------------
// Loop nests of the two templates, outer to inner.  Axis ids: GEMM i=0 j=1
// k=2; conv oc=0 oh=1 ow=2 rc=3 ry=4 rx=5.  FUSED marks the kernel-window
// loop r_l = (ry_l outer, rx_l inner).  Binding ids follow the annotation
// column: 3/4/5 blockIdx.x/y/z, 6/7/8 threadIdx.x/y/z, 0 serial.  The
// spatial axes (the first SPATIAL) are those whose third tiling level a
// vthread knob binds to virtual threads (id 9); a vectorize knob marks the
// innermost loop vectorized (id 10).
// --------------------------------------------------------------------------
constexpr int FUSED = -1;
constexpr uint32_t ANN_VTHREAD = 9u, ANN_VECTORIZE = 10u;
constexpr int ANN_KINDS = 12;   // one-hot annotation columns (ids 0 .. 11)

template <int TMPL> struct Nest;

template <> struct Nest<AT_TMPL_GEMM> {
    static constexpr int L = 10;
    static constexpr int F = 110;
    static constexpr int axis[L] = {0, 1, 0, 1, 2, 0, 1, 2, 0, 1};
    static constexpr int level[L] = {0, 0, 1, 1, 0, 2, 2, 1, 3, 3};
    static constexpr int bind[L] = {4, 3, 7, 6, 0, 0, 0, 0, 0, 0};
    static constexpr int SPATIAL = 2;
    // touch counts from the per-axis ranges of a sub-nest
    __device__ static void touched(const uint32_t (&r)[6], uint32_t, uint32_t (&t)[3]) {
        t[0] = r[2] * r[0];   // A[k][i]
        t[1] = r[2] * r[1];   // B[k][j]
        t[2] = r[0] * r[1];   // C[i][j]
    }
};

template <> struct Nest<AT_TMPL_CONV2D_NCHW> {
    static constexpr int L = 16;
    static constexpr int F = 176;
    static constexpr int axis[L] = {0, 1, 2, 0, 1, 2, 3, FUSED, 0, 1, 2, 3, FUSED, 0, 1, 2};
    static constexpr int level[L] = {0, 0, 0, 1, 1, 1, 0, 0, 2, 2, 2, 1, 1, 3, 3, 3};
    static constexpr int bind[L] = {5, 4, 3, 8, 7, 6, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
    static constexpr int SPATIAL = 3;
    __device__ static void touched(const uint32_t (&r)[6], uint32_t S, uint32_t (&t)[3]) {
        // data_pad[rc][oh*S+ry][ow*S+rx], unclipped padded coordinates
        t[0] = r[3] * distinct_affine(r[1], r[4], S) * distinct_affine(r[2], r[5], S);
        t[1] = r[0] * r[3] * r[4] * r[5];   // kernel[oc][rc][ry][rx]
        t[2] = r[0] * r[1] * r[2];          // output[oc][oh][ow]
    }
};

// Annotation id of loop p: its thread or block binding, else virtual
// threads (vth set, third level of a spatial axis), else vectorized (vec set,
// innermost loop), else unrolled (id unroll_id) when auto_unroll_max_step is
// on and its sub-nest has at most that many iterations, else serial.
template <int TMPL>
__device__ __forceinline__ uint32_t annotation_of(int p, uint32_t bottom_up, uint32_t unroll_max, uint32_t unroll_id,
                                                  uint32_t vec, uint32_t vth) {
    using N = Nest<TMPL>;
    if (N::bind[p]) return (uint32_t)N::bind[p];
    if (vth && N::level[p] == 2 && N::axis[p] >= 0 && N::axis[p] < N::SPATIAL) return ANN_VTHREAD;
    if (vec && p == N::L - 1) return ANN_VECTORIZE;
    return (unroll_max > 0u && bottom_up <= unroll_max) ? unroll_id : 0u;
}

// The annotation knobs of configuration kv: auto_unroll_max_step,
// unroll_explicit (id 1 or 2 for unrolled loops) and, for the annotated
// templates, vectorize and vthread.
struct AnnKnobs {
    uint32_t unroll_max, unroll_id, vec, vth;
};
template <int TMPL>
__device__ __forceinline__ AnnKnobs ann_knobs_of(const SpaceDesc& sd, const uint32_t (&kv)[MAX_KNOBS]) {
    constexpr int A = (TMPL == AT_TMPL_GEMM) ? 3 : 6;
    AnnKnobs k;
    k.unroll_max = kv[A] == 0u ? 0u : (kv[A] == 1u ? 512u : 1500u);
    k.unroll_id = 1u + kv[A + 1];
    k.vec = sd.ann_knobs ? kv[A + 2] : 0u;
    k.vth = sd.ann_knobs ? kv[A + 3] : 0u;
    return k;
}

// Factors of the chosen split of axis a: four 16-bit fields, outer level first.
__device__ __forceinline__ void unpack_split(uint64_t w, uint32_t (&f)[4]) {
    f[0] = (uint32_t)(w & 0xffff);
    f[1] = (uint32_t)((w >> 16) & 0xffff);
    f[2] = (uint32_t)((w >> 32) & 0xffff);
    f[3] = (uint32_t)(w >> 48);
}

// Loop-context features of one schedule.  The nest is walked from the
// innermost loop outwards so that each loop's sub-nest quantities are running
// products: range[a] is the extent of axis a covered by the sub-nest, and a
// loop's stride in buffer b is b's weight of the loop's axis times the range
// of that axis strictly inside the loop.  emit(f, value) receives feature f.
// PER = 13 gives the full rows of Appendix A.2: bitlen(top-down) and
// bitlen(bottom-up) follow the annotation.  Top-down is the nest's iteration
// count (the product of every factor, below 2^31 for any space) divided by
// bottom-up, the quotient's bitlen taken without a division.  PER = 24 gives
// the full rows with the annotation one-hot: ANN_KINDS columns, 1 at the
// loop's annotation id, 0 elsewhere.
template <int TMPL, int PER = 11, class Emit>
__device__ __forceinline__ void nest_features(const SpaceDesc& sd, const uint32_t (&fac)[6][4], const AnnKnobs& ak,
                                              Emit&& emit) {
    static_assert(PER == 11 || PER == 13 || PER == 24, "loop-context rows, full rows or one-hot rows");
    using N = Nest<TMPL>;
    constexpr int HOT = PER == 24 ? ANN_KINDS : 1;          // annotation columns
    constexpr int B0 = 1 + HOT + (PER == 11 ? 0 : 2);       // first buffer column
    uint32_t range[6] = {1u, 1u, 1u, 1u, 1u, 1u};
    uint32_t bottom_up = 1u;
    const uint32_t S = (uint32_t)sd.stride;
    uint32_t total = 1u;
    if constexpr (PER != 11) {
#pragma unroll
        for (int a = 0; a < 6; ++a)
#pragma unroll
            for (int l = 0; l < 4; ++l) total *= fac[a][l];
    }
#pragma unroll
    for (int p = N::L - 1; p >= 0; --p) {
        uint32_t ext, strd[3];
        if (N::axis[p] == FUSED) {
            const int l = N::level[p];
            const uint32_t fy = fac[4][l], fx = fac[5][l];
            ext = fy * fx;
            // one step of r moves rx when rx has several values, else ry
#pragma unroll
            for (int b = 0; b < 3; ++b)
                strd[b] = (fx > 1u) ? (uint32_t)sd.coef[b][5] * range[5] : (uint32_t)sd.coef[b][4] * range[4];
            range[4] *= fy;
            range[5] *= fx;
        } else {
            const int a = N::axis[p];
            ext = fac[a][N::level[p]];
#pragma unroll
            for (int b = 0; b < 3; ++b) strd[b] = (uint32_t)sd.coef[b][a] * range[a];
            range[a] *= ext;
        }
        bottom_up *= ext;
        uint32_t t[3];
        N::touched(range, S, t);
        const uint32_t ann = annotation_of<TMPL>(p, bottom_up, ak.unroll_max, ak.unroll_id, ak.vec, ak.vth);
        emit(p * PER + 0, bitlen(ext));
        if constexpr (PER == 24) {
#pragma unroll
            for (int h = 0; h < ANN_KINDS; ++h) emit(p * PER + 1 + h, ann == (uint32_t)h ? 1u : 0u);
        } else {
            emit(p * PER + 1, ann);
        }
        if constexpr (PER != 11) {
            emit(p * PER + 1 + HOT, bitlen_quot(total, bottom_up));
            emit(p * PER + 2 + HOT, bitlen(bottom_up));
        }
#pragma unroll
        for (int b = 0; b < 3; ++b) {
            emit(p * PER + B0 + 3 * b, bitlen(t[b]));
            emit(p * PER + B0 + 1 + 3 * b, bitlen_quot(bottom_up, t[b]));
            emit(p * PER + B0 + 2 + 3 * b, bitlen(strd[b]));
        }
    }
}

// The loop-context features of loop p alone (out[0..10]), for evaluating one
// schedule with one lane per loop.  Same arithmetic as nest_features: the
// running products over the loops at or inside p are formed by visiting every
// loop from the innermost outwards and multiplying in only those with index
// >= p; loop p's own quantities are captured when it is visited.  td, when
// given, receives bitlen(top-down) of loop p: the product of the lengths of
// the loops outside it, i.e. the nest's iteration count over bottom-up.
template <int TMPL>
__device__ __forceinline__ void loop_features(const SpaceDesc& sd, const uint32_t (&fac)[6][4], const AnnKnobs& ak,
                                              int p, uint32_t (&out)[11], uint32_t* td = nullptr) {
    using N = Nest<TMPL>;
    uint32_t range[6] = {1u, 1u, 1u, 1u, 1u, 1u};
    uint32_t bottom_up = 1u, ext = 1u;
    uint32_t strd[3] = {0u, 0u, 0u};
#pragma unroll
    for (int q = N::L - 1; q >= 0; --q) {
        const bool in = q >= p, at = q == p;
        uint32_t e, sq[3];
        if (N::axis[q] == FUSED) {
            const int l = N::level[q];
            const uint32_t fy = fac[4][l], fx = fac[5][l];
            e = fy * fx;
#pragma unroll
            for (int b = 0; b < 3; ++b)
                sq[b] = (fx > 1u) ? (uint32_t)sd.coef[b][5] * range[5] : (uint32_t)sd.coef[b][4] * range[4];
            range[4] *= in ? fy : 1u;
            range[5] *= in ? fx : 1u;
        } else {
            const int a = N::axis[q];
            e = fac[a][N::level[q]];
#pragma unroll
            for (int b = 0; b < 3; ++b) sq[b] = (uint32_t)sd.coef[b][a] * range[a];
            range[a] *= in ? e : 1u;
        }
        bottom_up *= in ? e : 1u;
        if (at) {
            ext = e;
#pragma unroll
            for (int b = 0; b < 3; ++b) strd[b] = sq[b];
        }
    }
    uint32_t t[3];
    N::touched(range, (uint32_t)sd.stride, t);
    if (td) {
        uint32_t total = 1u;
#pragma unroll
        for (int a = 0; a < 6; ++a)
#pragma unroll
            for (int l = 0; l < 4; ++l) total *= fac[a][l];
        *td = bitlen_quot(total, bottom_up);
    }
    out[0] = bitlen(ext);
    out[1] = annotation_of<TMPL>(p, bottom_up, ak.unroll_max, ak.unroll_id, ak.vec, ak.vth);
#pragma unroll
    for (int b = 0; b < 3; ++b) {
        out[2 + 3 * b] = bitlen(t[b]);
        out[3 + 3 * b] = bitlen_quot(bottom_up, t[b]);
        out[4 + 3 * b] = bitlen(strd[b]);
    }
}


// Factors of every axis for knob values kv (split knob a = axis a).
template <int TMPL>
__device__ __forceinline__ void gather_factors(const SpaceDesc& sd, const uint64_t* __restrict__ factors,
                                               const uint32_t (&kv)[MAX_KNOBS], uint32_t (&fac)[6][4]) {
    constexpr int A = (TMPL == AT_TMPL_GEMM) ? 3 : 6;
#pragma unroll
    for (int a = 0; a < 6; ++a) {
        if (a < A) unpack_split(factors[sd.split_off[a] + kv[a]], fac[a]);
        else fac[a][0] = fac[a][1] = fac[a][2] = fac[a][3] = 1u;
    }
}

// Copies `words` packed tree words (a multiple of 4) from global to LDS.
__device__ __forceinline__ void stage_words(uint32_t* __restrict__ dst, const uint32_t* __restrict__ src,
                                            int words) {
    const uint4* s4 = reinterpret_cast<const uint4*>(src);
    uint4* d4 = reinterpret_cast<uint4*>(dst);
    for (int i = threadIdx.x; i < words / 4; i += WG) d4[i] = s4[i];
}

// Walks GROUP trees of depth DEPTH starting at chunk word `cb` (tree stride
// W words) for the lane whose feature column starts at byte `fb` of the
// tile; returns the leaf words and leaf indices.
template <int DEPTH, int GROUP>
__device__ __forceinline__ void walk(const uint32_t* __restrict__ chunk, const uint8_t* __restrict__ tile_b,
                                     uint32_t fb, int cb, uint32_t (&leafw)[GROUP], uint32_t (&leafi)[GROUP]) {
    constexpr int W = 2 << DEPTH;
    uint32_t m[GROUP];
#pragma unroll
    for (int g = 0; g < GROUP; ++g) m[g] = 1u;
#pragma unroll
    for (int l = 0; l < DEPTH; ++l) {
        uint32_t node[GROUP];
#pragma unroll
        for (int g = 0; g < GROUP; ++g) node[g] = chunk[cb + g * W + m[g]];
#pragma unroll
        for (int g = 0; g < GROUP; ++g) {
            const uint32_t x = tile_b[fb + (node[g] & 0xffffu)];
            m[g] = 2u * m[g] + (x >= (node[g] >> 16) ? 1u : 0u);
        }
    }
#pragma unroll
    for (int g = 0; g < GROUP; ++g) {
        leafw[g] = chunk[cb + g * W + m[g]];
        leafi[g] = m[g] - (1u << DEPTH);
    }
}

// Walks GROUP trees whose words start at byte tree_off (tree stride 4*W
// bytes) of the LDS block L, for the row whose feature column starts at byte
// fb of L.  One LDS round trip per level: the current node's feature byte and
// the pair of its children (words 2m, 2m+1, bytes 8m..8m+7) are read
// together and the child is then selected; at the last level the pair holds
// two leaves.  Returns the leaf words and leaf indices.
template <int DEPTH, int GROUP>
__device__ __forceinline__ void walk_pair(const uint8_t* __restrict__ L, uint32_t tree_off, uint32_t fb,
                                          uint32_t (&leafw)[GROUP], uint32_t (&leafi)[GROUP]) {
    constexpr uint32_t TB = (2u << DEPTH) * 4u;
    uint32_t node[GROUP], a[GROUP];
#pragma unroll
    for (int g = 0; g < GROUP; ++g) {
        node[g] = *reinterpret_cast<const uint32_t*>(L + tree_off + g * TB + 4u);
        a[g] = 8u;
    }
#pragma unroll
    for (int l = 0; l < DEPTH; ++l) {
        uint32_t x[GROUP];
        uint2 pr[GROUP];
#pragma unroll
        for (int g = 0; g < GROUP; ++g) {
            x[g] = L[fb + (node[g] & 0xffffu)];
            pr[g] = *reinterpret_cast<const uint2*>(L + tree_off + g * TB + a[g]);
        }
#pragma unroll
        for (int g = 0; g < GROUP; ++g) {
            const bool right = x[g] >= (node[g] >> 16);
            node[g] = right ? pr[g].y : pr[g].x;
            a[g] = 2u * a[g] + (right ? 8u : 0u);
        }
    }
#pragma unroll
    for (int g = 0; g < GROUP; ++g) {
        leafw[g] = node[g];
        leafi[g] = (a[g] >> 3) - (1u << DEPTH);
    }
}

}  // namespace dev
}  // namespace at
