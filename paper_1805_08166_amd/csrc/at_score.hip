// Batched ensemble scoring for conv2d feature rows: 176 loop-context
// features or 192 context relation features (44 or 48 feature quads).
//
// One candidate per lane, 256 per workgroup.  LDS holds one chunk of packed
// tree words (8 KB, 32 KB for depth 12) followed by the workgroup's feature
// tile (176 u8 per row, quad-major), 53 KB in all at depth 8 so that three
// workgroups share a compute unit.  The next chunk is fetched into registers
// while the current one is walked; the walk keeps GROUP trees in flight per
// lane and needs one LDS round trip per level (walk_pair).  Scores are the
// fp32 sum of the reached leaves in tree order, starting from +0.0f.
#include "at_device.h"

namespace at {
namespace {

using namespace dev;

constexpr int SWG = 256;

template <int DEPTH> struct ScoreShape {
    static constexpr int W = 2 << DEPTH;                       // words per tree
    static constexpr int CW = DEPTH <= 10 ? 2048 : (DEPTH == 11 ? 4096 : 8192);   // words per chunk
    static constexpr int CT = CW / W;                          // trees per chunk
    static constexpr int G = CT < 4 ? CT : 4;                  // trees walked together
    static constexpr int PER = CW / 4 / SWG;                   // 16-byte pieces per thread
};

template <int DEPTH, int GR, bool LEAVES>
__device__ __forceinline__ void walk_add(const uint8_t* L, uint32_t off, uint32_t fb, float& acc, uint16_t* lrow,
                                         int t_global) {
    uint32_t lw[GR], li[GR];
    walk_pair<DEPTH, GR>(L, off, fb, lw, li);
#pragma unroll
    for (int g = 0; g < GR; ++g) {
        acc = acc + __uint_as_float(lw[g]);
        // lanes past the last row have no output row (lrow is null)
        if (LEAVES && lrow) lrow[t_global + g] = (uint16_t)li[g];
    }
}

// walks r (< 2*H) remaining trees of a partial chunk in groups of H, H/2, ..., 1
template <int DEPTH, int H, bool LEAVES>
__device__ __forceinline__ void walk_add_rest(const uint8_t* L, int t, int r, uint32_t fb, float& acc,
                                              uint16_t* lrow, int t0) {
    constexpr uint32_t TB = (2u << DEPTH) * 4u;
    if (r >= H) {
        walk_add<DEPTH, H, LEAVES>(L, (uint32_t)t * TB, fb, acc, lrow, t0 + t);
        t += H;
        r -= H;
    }
    if constexpr (H > 1) walk_add_rest<DEPTH, H / 2, LEAVES>(L, t, r, fb, acc, lrow, t0);
}

// SQ: feature quads of a row (44 or 48); accumulate: add the score to the
// value already in scores (fp32, that value first) instead of storing it.
template <int DEPTH, bool LEAVES, int SQ>
__global__ __launch_bounds__(SWG) void k_score(EnsembleDesc e, const int32_t* __restrict__ feats, int64_t n,
                                               float* __restrict__ scores, uint16_t* __restrict__ leaves,
                                               int accumulate) {
    using S = ScoreShape<DEPTH>;
    constexpr int PK = SQ % 11 == 0 ? 11 : 12;   // quads loaded together
    constexpr uint32_t TB = (uint32_t)S::W * 4u;
    __shared__ uint32_t lds[S::CW + SQ * SWG];
    const uint8_t* L = reinterpret_cast<const uint8_t*>(lds);
    uint4* chunk4 = reinterpret_cast<uint4*>(lds);
    uint32_t* tile = lds + S::CW;
    const int tid = threadIdx.x;
    const int64_t row = (int64_t)blockIdx.x * SWG + tid;
    const uint4* src = reinterpret_cast<const uint4*>(e.words);

    // first chunk in flight while the feature row is packed into the tile
    uint32_t pre[S::PER * 4];
#pragma unroll
    for (int u = 0; u < S::PER; ++u) {
        const uint4 x = src[tid + u * SWG];
        pre[4 * u] = x.x; pre[4 * u + 1] = x.y; pre[4 * u + 2] = x.z; pre[4 * u + 3] = x.w;
    }
    {
        // rows past the end repeat the last row; their results are not stored
        const int64_t r = row < n ? row : n - 1;
        const int4* fr = reinterpret_cast<const int4*>(feats + r * (SQ * 4));
        uint32_t packed[SQ];
#pragma unroll
        for (int h = 0; h < SQ; h += PK) {
            int4 v[PK];
#pragma unroll
            for (int q = 0; q < PK; ++q) v[q] = fr[h + q];
#pragma unroll
            for (int q = 0; q < PK; ++q) {
                const uint32_t b0 = (uint32_t)min(max(v[q].x, 0), 255), b1 = (uint32_t)min(max(v[q].y, 0), 255);
                const uint32_t b2 = (uint32_t)min(max(v[q].z, 0), 255), b3 = (uint32_t)min(max(v[q].w, 0), 255);
                packed[h + q] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
            }
        }
#pragma unroll
        for (int q = 0; q < SQ; ++q) tile[q * SWG + tid] = packed[q];
    }
    const uint32_t fb = (uint32_t)S::CW * 4u + (uint32_t)tid * 4u;
    uint16_t* lrow = (LEAVES && row < n) ? leaves + row * e.n_trees : nullptr;
    float acc = 0.0f;
    const int nchunks = (e.n_trees + S::CT - 1) / S::CT;
    for (int k = 0; k < nchunks; ++k) {
        __syncthreads();
#pragma unroll
        for (int u = 0; u < S::PER; ++u)
            chunk4[tid + u * SWG] = make_uint4(pre[4 * u], pre[4 * u + 1], pre[4 * u + 2], pre[4 * u + 3]);
        __syncthreads();
        // next chunk (the last one is fetched again on the final pass; the
        // packed ensemble is padded so every fetch stays in bounds)
        const int kn = (k + 1 < nchunks) ? k + 1 : k;
        const uint4* s4 = src + (size_t)kn * (S::CW / 4);
#pragma unroll
        for (int u = 0; u < S::PER; ++u) {
            const uint4 x = s4[tid + u * SWG];
            pre[4 * u] = x.x; pre[4 * u + 1] = x.y; pre[4 * u + 2] = x.z; pre[4 * u + 3] = x.w;
        }
        const int t0 = k * S::CT;
        const int nt = (e.n_trees - t0 < S::CT) ? e.n_trees - t0 : S::CT;
        if (nt == S::CT) {
#pragma unroll 4
            for (int t = 0; t < S::CT; t += S::G)
                walk_add<DEPTH, S::G, LEAVES>(L, (uint32_t)t * TB, fb, acc, lrow, t0 + t);
        } else {
            int t = 0;
            for (; t + S::G <= nt; t += S::G)
                walk_add<DEPTH, S::G, LEAVES>(L, (uint32_t)t * TB, fb, acc, lrow, t0 + t);
            if constexpr (S::G > 1) walk_add_rest<DEPTH, S::G / 2, LEAVES>(L, t, nt - t, fb, acc, lrow, t0);
        }
    }
    if (row < n) scores[row] = accumulate ? scores[row] + acc : acc;
}

template <int DEPTH, int SQ>
hipError_t score_q(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves,
                   bool accumulate, hipStream_t stream) {
    const unsigned grid = (unsigned)((n + SWG - 1) / SWG);
    if (leaves)
        hipLaunchKernelGGL((k_score<DEPTH, true, SQ>), dim3(grid), dim3(SWG), 0, stream, e, feats, n, scores, leaves,
                           accumulate ? 1 : 0);
    else
        hipLaunchKernelGGL((k_score<DEPTH, false, SQ>), dim3(grid), dim3(SWG), 0, stream, e, feats, n, scores, leaves,
                           accumulate ? 1 : 0);
    return hipGetLastError();
}

template <int DEPTH>
hipError_t score_depth(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves,
                       bool accumulate, hipStream_t stream) {
    if (e.n_features == 192) return score_q<DEPTH, 48>(e, feats, n, scores, leaves, accumulate, stream);
    return score_q<DEPTH, 44>(e, feats, n, scores, leaves, accumulate, stream);
}

}  // namespace

hipError_t launch_score(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves,
                        bool accumulate, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    switch (e.depth) {
        case 1: return score_depth<1>(e, feats, n, scores, leaves, accumulate, stream);
        case 2: return score_depth<2>(e, feats, n, scores, leaves, accumulate, stream);
        case 3: return score_depth<3>(e, feats, n, scores, leaves, accumulate, stream);
        case 4: return score_depth<4>(e, feats, n, scores, leaves, accumulate, stream);
        case 5: return score_depth<5>(e, feats, n, scores, leaves, accumulate, stream);
        case 6: return score_depth<6>(e, feats, n, scores, leaves, accumulate, stream);
        case 7: return score_depth<7>(e, feats, n, scores, leaves, accumulate, stream);
        case 8: return score_depth<8>(e, feats, n, scores, leaves, accumulate, stream);
        case 9: return score_depth<9>(e, feats, n, scores, leaves, accumulate, stream);
        case 10: return score_depth<10>(e, feats, n, scores, leaves, accumulate, stream);
        case 11: return score_depth<11>(e, feats, n, scores, leaves, accumulate, stream);
        case 12: return score_depth<12>(e, feats, n, scores, leaves, accumulate, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace at
