// HIP kernels for gfx950 (CDNA4): loop-context features, tree-ensemble
// scoring and parallel simulated annealing.
//
// Nothing here is a dense contraction, so there is no MFMA: the features are
// integer bookkeeping bound by HBM writes, and the tree walk is a chain of
// dependent LDS gathers bound by LDS and VALU issue.
//
// Exactness: features are integers; a score is the fp32 sum of the reached
// leaves added one tree after another in tree order from +0.0f, exactly as
// the model defines it, so every kernel reproduces it bit for bit.  The
// library is compiled with -ffp-contract=off.
#include "at_device.h"

namespace at {
namespace {

using namespace dev;

// ==========================================================================
// Feature extraction: one configuration per lane.  Rows are built as signed
// bytes in LDS (row stride with an odd dword count so the per-lane byte
// writes spread over the banks) and then written out as int32 with
// consecutive lanes covering consecutive 16-byte pieces of the block, so the
// HBM stores are fully coalesced.
// ==========================================================================
// PER columns per loop: 11 (loop-context rows), 13 (full Appendix A.2 rows
// with top-down and bottom-up) or 24 (full rows with a one-hot annotation)
template <int TMPL, int PER = 11>
struct RowLayout {
    static constexpr int F = Nest<TMPL>::L * PER;
    static constexpr int RS = ((F + 3) / 4 % 2 == 1) ? ((F + 3) / 4) * 4 : ((F + 3) / 4 + 1) * 4;
};

template <int TMPL, bool VEC, int PER = 11>
__global__ __launch_bounds__(WG) void k_extract(SpaceDesc sd, const uint64_t* __restrict__ factors,
                                                const uint64_t* __restrict__ cfgs, int64_t n,
                                                int32_t* __restrict__ feats,
                                                unsigned long long* __restrict__ n_bad) {
    constexpr int F = RowLayout<TMPL, PER>::F;
    constexpr int RS = RowLayout<TMPL, PER>::RS;
    __shared__ int8_t rows[WG * RS];
    const int tid = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * WG;
    const int64_t row = base + tid;
    int8_t* my = rows + tid * RS;
    if (row < n) {
        const uint64_t cfg = cfgs[row];
        if (cfg >= sd.n_configs) {
            for (int f = 0; f < F; ++f) my[f] = -1;
            atomicAdd(n_bad, 1ull);
        } else {
            // mixed radix, knob 0 most significant; indices fit 32 bits
            uint32_t rest = (uint32_t)cfg;
            uint32_t kv[MAX_KNOBS];
#pragma unroll
            for (int j = MAX_KNOBS - 1; j >= 0; --j) {
                if (j < sd.n_knobs) {
                    const uint32_t sz = sd.knob_size[j];
                    const uint32_t q = rest / sz;
                    kv[j] = rest - q * sz;
                    rest = q;
                } else {
                    kv[j] = 0u;
                }
            }
            uint32_t fac[6][4];
            gather_factors<TMPL>(sd, factors, kv, fac);
            nest_features<TMPL, PER>(sd, fac, ann_knobs_of<TMPL>(sd, kv),
                                     [&](int f, uint32_t v) { my[f] = (int8_t)v; });
        }
    }
    __syncthreads();
    const int64_t rows_here = (n - base < WG) ? (n - base) : WG;
    const int total = (int)rows_here * F;
    int32_t* out = feats + base * F;
    if (VEC) {
        // F % 4 == 0: each thread moves 4 consecutive features of one row
        for (int g = tid; g < total / 4; g += WG) {
            const int e = g * 4;
            const int r = e / F, c = e - r * F;
            const int w = *reinterpret_cast<const int*>(rows + r * RS + c);
            int4 v;
            v.x = (int)(int8_t)(w & 0xff);
            v.y = (int)(int8_t)((w >> 8) & 0xff);
            v.z = (int)(int8_t)((w >> 16) & 0xff);
            v.w = (int)(int8_t)((w >> 24) & 0xff);
            *reinterpret_cast<int4*>(out + e) = v;
        }
    } else {
        for (int e = tid; e < total; e += WG) {
            const int r = e / F, c = e - r * F;
            out[e] = (int32_t)rows[r * RS + c];
        }
    }
}

// ==========================================================================
// Context relation features (Section 4; Appendix A.2), one configuration per
// lane.  Per buffer b and t = 1..REL_T, over the loops whose sub-nest
// touches fewer than 2^t elements of b (bitlen(touch) <= t):
//   R[0][b][t-1] = the largest bitlen(reuse ratio),
//   R[1][b][t-1] = the largest bitlen(top-down product of the outer lengths),
// 0 when no loop qualifies.  The loop quantities come from nest_features; the
// rows go through LDS as bytes (odd dword stride) to coalesced int4 stores.
// ==========================================================================
constexpr int REL_T = 32;
constexpr int REL_F = 2 * 3 * REL_T;        // 192 features per row
constexpr int REL_RS = REL_F + 4;           // 49 dwords per LDS row

template <int TMPL>
__global__ __launch_bounds__(WG) void k_relation(SpaceDesc sd, const uint64_t* __restrict__ factors,
                                                 const uint64_t* __restrict__ cfgs, int64_t n,
                                                 int32_t* __restrict__ feats, unsigned long long* __restrict__ n_bad) {
    using N = Nest<TMPL>;
    __shared__ int8_t rows[WG * REL_RS];
    const int tid = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * WG;
    const int64_t row = base + tid;
    int8_t* my = rows + tid * REL_RS;
    if (row < n) {
        const uint64_t cfg = cfgs[row];
        if (cfg >= sd.n_configs) {
            for (int f = 0; f < REL_F; ++f) my[f] = -1;
            atomicAdd(n_bad, 1ull);
        } else {
            uint32_t rest = (uint32_t)cfg;
            uint32_t kv[MAX_KNOBS];
#pragma unroll
            for (int j = MAX_KNOBS - 1; j >= 0; --j) {
                if (j < sd.n_knobs) {
                    const uint32_t sz = sd.knob_size[j];
                    const uint32_t q = rest / sz;
                    kv[j] = rest - q * sz;
                    rest = q;
                } else {
                    kv[j] = 0u;
                }
            }
            uint32_t fac[6][4];
            gather_factors<TMPL>(sd, factors, kv, fac);
            // per loop: bitlen of the touch count (tc) and of the reuse ratio (ru) per buffer
            uint32_t tc[N::L][3], ru[N::L][3];
            nest_features<TMPL>(sd, fac, ann_knobs_of<TMPL>(sd, kv), [&](int f, uint32_t v) {
                const int p = f / 11, c = f - p * 11;
                if (c >= 2 && (c - 2) % 3 == 0) tc[p][(c - 2) / 3] = v;
                if (c >= 2 && (c - 2) % 3 == 1) ru[p][(c - 2) / 3] = v;
            });
            // bitlen of the top-down product of each loop (outer lengths only)
            uint32_t td[N::L];
            uint32_t prod = 1u;
#pragma unroll
            for (int p = 0; p < N::L; ++p) {
                td[p] = bitlen(prod);
                const uint32_t e = N::axis[p] == FUSED ? fac[4][N::level[p]] * fac[5][N::level[p]]
                                                       : fac[N::axis[p]][N::level[p]];
                prod *= e;
            }
            // A sub-nest touches no fewer elements than any sub-nest inside
            // it, so the loops a threshold t admits (bitlen(touch) <= t) are
            // the innermost ones from some loop p* on, and each maximum is a
            // suffix maximum (over p* and the loops inside it).  Visiting the
            // loops from the innermost outwards, loop p writes its suffix
            // maxima into every threshold it admits; the outermost admitted
            // loop, p*, writes last.  Four thresholds share a word: byte j of
            // word w is t = 4w + 1 + j, admitted when j >= bitlen(touch) - 1 - 4w.
#pragma unroll
            for (int b = 0; b < 3; ++b) {
                constexpr int NW = REL_T / 4;
                uint32_t w0[NW], w1[NW];
#pragma unroll
                for (int w = 0; w < NW; ++w) w0[w] = w1[w] = 0u;
                uint32_t s0 = 0u, s1 = 0u;
#pragma unroll
                for (int p = N::L - 1; p >= 0; --p) {
                    s0 = max(s0, ru[p][b]);
                    s1 = max(s1, td[p]);
                    const uint32_t b0 = s0 * 0x01010101u, b1 = s1 * 0x01010101u;
#pragma unroll
                    for (int w = 0; w < NW; ++w) {
                        const int kb = min(max((int)tc[p][b] - 1 - 4 * w, 0), 4);
                        const uint32_t m = (uint32_t)(0xffffffffull << (8 * kb));
                        w0[w] = (b0 & m) | (w0[w] & ~m);
                        w1[w] = (b1 & m) | (w1[w] & ~m);
                    }
                }
                // rows are dword aligned (REL_RS = 196 bytes) and so is each
                // 32-byte block
                uint32_t* d0 = reinterpret_cast<uint32_t*>(my + (0 * 3 + b) * REL_T);
                uint32_t* d1 = reinterpret_cast<uint32_t*>(my + (1 * 3 + b) * REL_T);
#pragma unroll
                for (int w = 0; w < NW; ++w) {
                    d0[w] = w0[w];
                    d1[w] = w1[w];
                }
            }
        }
    }
    __syncthreads();
    const int64_t rows_here = (n - base < WG) ? (n - base) : WG;
    const int total = (int)rows_here * REL_F;
    int32_t* out = feats + base * REL_F;
    for (int g = tid; g < total / 4; g += WG) {
        const int e = g * 4;
        const int r = e / REL_F, c = e - r * REL_F;
        const int w = *reinterpret_cast<const int*>(rows + r * REL_RS + c);
        int4 v;
        v.x = (int)(int8_t)(w & 0xff);
        v.y = (int)(int8_t)((w >> 8) & 0xff);
        v.z = (int)(int8_t)((w >> 16) & 0xff);
        v.w = (int)(int8_t)((w >> 24) & 0xff);
        *reinterpret_cast<int4*>(out + e) = v;
    }
}

// ==========================================================================
// Tree-ensemble traversal shared by scoring and annealing.
// A workgroup holds the features of its 256 rows (chains or candidates) in
// an LDS tile and streams the packed trees through LDS in chunks.  Each lane
// walks every tree for its own row and adds the leaves in tree order.
// ==========================================================================

// Scores the row in this lane's tile column against every tree; all lanes
// of the workgroup must call it together (it stages chunks with barriers).
template <int DEPTH>
__device__ __forceinline__ float score_tile(const EnsembleDesc& e, const uint32_t* __restrict__ tile, uint32_t* __restrict__ chunk,
                            int chunk_trees, uint16_t* __restrict__ leaves_row) {
    constexpr int W = 2 << DEPTH;
    constexpr int G = 4;
    const uint8_t* tile_b = reinterpret_cast<const uint8_t*>(tile);
    const uint32_t fb = threadIdx.x * 4u;
    float acc = 0.0f;
    for (int t0 = 0; t0 < e.n_trees; t0 += chunk_trees) {
        const int nt = (e.n_trees - t0 < chunk_trees) ? (e.n_trees - t0) : chunk_trees;
        __syncthreads();
        stage_words(chunk, e.words + (size_t)t0 * W, nt * W);
        __syncthreads();
        int t = 0;
        for (; t + G <= nt; t += G) {
            uint32_t lw[G], li[G];
            walk<DEPTH, G>(chunk, tile_b, fb, t * W, lw, li);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                acc = acc + __uint_as_float(lw[g]);
                if (leaves_row) leaves_row[t0 + t + g] = (uint16_t)li[g];
            }
        }
        for (; t < nt; ++t) {
            uint32_t lw[1], li[1];
            walk<DEPTH, 1>(chunk, tile_b, fb, t * W, lw, li);
            acc = acc + __uint_as_float(lw[0]);
            if (leaves_row) leaves_row[t0 + t] = (uint16_t)li[0];
        }
    }
    return acc;
}

// Trees per LDS chunk: the largest count whose words fit `bytes`.
__host__ __device__ inline int chunk_trees_for(int depth, int bytes) {
    int w = 2 << depth;
    int t = bytes / (w * 4);
    return t < 1 ? 1 : t;
}

constexpr int CHUNK_BYTES = 32768;

template <int DEPTH>
__global__ __launch_bounds__(WG) void k_predict(EnsembleDesc e, const int32_t* __restrict__ feats, int64_t n,
                                                float* __restrict__ scores, uint16_t* __restrict__ leaves,
                                                int chunk_trees, int accumulate) {
    extern __shared__ uint32_t lds[];
    const int Q = (e.n_features + 3) / 4;
    uint32_t* tile = lds;
    uint32_t* chunk = lds + Q * WG;
    const int tid = threadIdx.x;
    const int64_t row = (int64_t)blockIdx.x * WG + tid;
    const int F = e.n_features;
    // own row -> tile column, 4 features per dword, clamped to [0, 255]
    for (int q = 0; q < Q; ++q) {
        uint32_t w = 0;
        if (row < n) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int f = q * 4 + k;
                if (f < F) {
                    int x = feats[row * F + f];
                    x = x < 0 ? 0 : (x > 255 ? 255 : x);
                    w |= (uint32_t)x << (8 * k);
                }
            }
        }
        tile[q * WG + tid] = w;
    }
    uint16_t* lrow = (leaves && row < n) ? leaves + row * e.n_trees : nullptr;
    const float s = score_tile<DEPTH>(e, tile, chunk, chunk_trees, lrow);
    if (row < n) scores[row] = accumulate ? scores[row] + s : s;
}

__global__ __launch_bounds__(WG) void k_export(const SpaceDesc* descs, const int64_t* offsets, int n_spaces,
                                               const uint16_t* knobs, const float* score, int64_t n,
                                               uint64_t* cur_cfg, float* cur_score) {
    const int64_t c = (int64_t)blockIdx.x * WG + threadIdx.x;
    if (c >= n) return;
    int w = 0;
    while (w + 1 < n_spaces && offsets[w + 1] <= c) ++w;
    const SpaceDesc& sd = descs[w];
    if (cur_cfg) {
        uint64_t x = 0;
        for (int j = 0; j < sd.n_knobs; ++j) x += (uint64_t)knobs[c * MAX_KNOBS + j] * sd.radix[j];
        cur_cfg[c] = x;
    }
    if (cur_score) cur_score[c] = score[c];
}

// ==========================================================================
// Which loop-context features are constant over a space.  Every
// configuration index below n is visited (grid-stride loop, one per lane);
// flags[f] becomes 1 when some configuration's feature f differs from that
// of configuration 0, and workgroup 0 writes configuration 0's row to ref.
// A feature left unflagged therefore takes one value over the whole space.
// ==========================================================================
template <int TMPL>
__global__ __launch_bounds__(WG) void k_feature_scan(SpaceDesc sd, const uint64_t* __restrict__ factors, uint64_t n,
                                                     uint32_t* __restrict__ flags, uint32_t* __restrict__ ref_out) {
    constexpr int F = RowLayout<TMPL>::F;
    __shared__ uint32_t ref[F];
    __shared__ uint32_t diff[F];
    const int tid = threadIdx.x;
    auto row_of = [&](uint64_t cfg, auto&& put) {
        // mixed radix, knob 0 most significant (indices below n fit 32 bits)
        uint32_t rest = (uint32_t)cfg;
        uint32_t kv[MAX_KNOBS];
#pragma unroll
        for (int j = MAX_KNOBS - 1; j >= 0; --j) {
            if (j < sd.n_knobs) {
                const uint32_t sz = sd.knob_size[j];
                const uint32_t q = rest / sz;
                kv[j] = rest - q * sz;
                rest = q;
            } else {
                kv[j] = 0u;
            }
        }
        uint32_t fac[6][4];
        gather_factors<TMPL>(sd, factors, kv, fac);
        nest_features<TMPL, 11>(sd, fac, ann_knobs_of<TMPL>(sd, kv), put);
    };
    for (int f = tid; f < F; f += WG) diff[f] = 0u;
    if (tid == 0) row_of(0, [&](int f, uint32_t v) { ref[f] = v; });
    __syncthreads();
    const uint64_t stride = (uint64_t)gridDim.x * WG;
    for (uint64_t cfg = (uint64_t)blockIdx.x * WG + tid; cfg < n; cfg += stride)
        row_of(cfg, [&](int f, uint32_t v) {
            if (v != ref[f]) diff[f] = 1u;
        });
    __syncthreads();
    for (int f = tid; f < F; f += WG) {
        if (diff[f]) flags[f] = 1u;
        if (blockIdx.x == 0) ref_out[f] = ref[f];
    }
}

}  // namespace

hipError_t launch_extract(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                          hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const SpaceDesc& sd = sp.descs[0];
    const unsigned grid = (unsigned)((n + WG - 1) / WG);
    const uint64_t* fac = static_cast<const uint64_t*>(sp.d_factors.p);
    auto* bad = static_cast<unsigned long long*>(sp.d_errors.p);
    const bool aligned = (reinterpret_cast<uintptr_t>(feats) & 15u) == 0;
    if (sp.tmpl == AT_TMPL_GEMM) {
        // 110 features per row: not a multiple of 4, scalar stores
        hipLaunchKernelGGL((k_extract<AT_TMPL_GEMM, false>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs, n,
                           feats, bad);
    } else if (aligned) {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, true>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs,
                           n, feats, bad);
    } else {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, false>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs,
                           n, feats, bad);
    }
    return hipGetLastError();
}

hipError_t launch_extract_full(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                               hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const SpaceDesc& sd = sp.descs[0];
    const unsigned grid = (unsigned)((n + WG - 1) / WG);
    const uint64_t* fac = static_cast<const uint64_t*>(sp.d_factors.p);
    auto* bad = static_cast<unsigned long long*>(sp.d_errors.p);
    const bool aligned = (reinterpret_cast<uintptr_t>(feats) & 15u) == 0;
    if (sp.tmpl == AT_TMPL_GEMM) {
        // 130 features per row: not a multiple of 4, scalar stores
        hipLaunchKernelGGL((k_extract<AT_TMPL_GEMM, false, 13>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs, n,
                           feats, bad);
    } else if (aligned) {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, true, 13>), dim3(grid), dim3(WG), 0, stream, sd, fac,
                           cfgs, n, feats, bad);
    } else {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, false, 13>), dim3(grid), dim3(WG), 0, stream, sd, fac,
                           cfgs, n, feats, bad);
    }
    return hipGetLastError();
}

hipError_t launch_extract_onehot(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                 hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const SpaceDesc& sd = sp.descs[0];
    const unsigned grid = (unsigned)((n + WG - 1) / WG);
    const uint64_t* fac = static_cast<const uint64_t*>(sp.d_factors.p);
    auto* bad = static_cast<unsigned long long*>(sp.d_errors.p);
    const bool aligned = (reinterpret_cast<uintptr_t>(feats) & 15u) == 0;
    // 240 (GEMM) and 384 (conv2d) features per row, both multiples of 4
    if (sp.tmpl == AT_TMPL_GEMM) {
        if (aligned)
            hipLaunchKernelGGL((k_extract<AT_TMPL_GEMM, true, 24>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs, n,
                               feats, bad);
        else
            hipLaunchKernelGGL((k_extract<AT_TMPL_GEMM, false, 24>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs,
                               n, feats, bad);
    } else if (aligned) {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, true, 24>), dim3(grid), dim3(WG), 0, stream, sd, fac,
                           cfgs, n, feats, bad);
    } else {
        hipLaunchKernelGGL((k_extract<AT_TMPL_CONV2D_NCHW, false, 24>), dim3(grid), dim3(WG), 0, stream, sd, fac,
                           cfgs, n, feats, bad);
    }
    return hipGetLastError();
}

hipError_t launch_relation(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                           hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const SpaceDesc& sd = sp.descs[0];
    const unsigned grid = (unsigned)((n + WG - 1) / WG);
    const uint64_t* fac = static_cast<const uint64_t*>(sp.d_factors.p);
    auto* bad = static_cast<unsigned long long*>(sp.d_errors.p);
    if (sp.tmpl == AT_TMPL_GEMM)
        hipLaunchKernelGGL((k_relation<AT_TMPL_GEMM>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs, n, feats, bad);
    else
        hipLaunchKernelGGL((k_relation<AT_TMPL_CONV2D_NCHW>), dim3(grid), dim3(WG), 0, stream, sd, fac, cfgs, n,
                           feats, bad);
    return hipGetLastError();
}

namespace {

template <int DEPTH>
hipError_t predict_depth(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves,
                         bool accumulate, hipStream_t stream) {
    const int Q = (e.n_features + 3) / 4;
    const int ct = chunk_trees_for(DEPTH, CHUNK_BYTES);
    const size_t lds = (size_t)Q * WG * 4 + (size_t)ct * (2 << DEPTH) * 4;
    hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_predict<DEPTH>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (err != hipSuccess) return err;
    const unsigned grid = (unsigned)((n + WG - 1) / WG);
    hipLaunchKernelGGL((k_predict<DEPTH>), dim3(grid), dim3(WG), lds, stream, e, feats, n, scores, leaves, ct,
                       accumulate ? 1 : 0);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_predict(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores,
                          uint16_t* leaves, bool accumulate, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    // conv2d loop-feature rows (176) and relation-feature rows (192), 16-byte
    // aligned, take the tuned kernel
    if ((e.n_features == 176 || e.n_features == 192) && (reinterpret_cast<uintptr_t>(feats) & 15u) == 0)
        return launch_score(e, feats, n, scores, leaves, accumulate, stream);
    switch (e.depth) {
        case 1: return predict_depth<1>(e, feats, n, scores, leaves, accumulate, stream);
        case 2: return predict_depth<2>(e, feats, n, scores, leaves, accumulate, stream);
        case 3: return predict_depth<3>(e, feats, n, scores, leaves, accumulate, stream);
        case 4: return predict_depth<4>(e, feats, n, scores, leaves, accumulate, stream);
        case 5: return predict_depth<5>(e, feats, n, scores, leaves, accumulate, stream);
        case 6: return predict_depth<6>(e, feats, n, scores, leaves, accumulate, stream);
        case 7: return predict_depth<7>(e, feats, n, scores, leaves, accumulate, stream);
        case 8: return predict_depth<8>(e, feats, n, scores, leaves, accumulate, stream);
        case 9: return predict_depth<9>(e, feats, n, scores, leaves, accumulate, stream);
        case 10: return predict_depth<10>(e, feats, n, scores, leaves, accumulate, stream);
        case 11: return predict_depth<11>(e, feats, n, scores, leaves, accumulate, stream);
        case 12: return predict_depth<12>(e, feats, n, scores, leaves, accumulate, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_feature_scan(const at_space_s& sp, uint32_t* flags, uint32_t* ref, hipStream_t stream) {
    const SpaceDesc& sd = sp.descs[0];
    const uint64_t n = sd.n_configs;
    if (n == 0) return hipSuccess;
    const uint64_t blocks = (n + WG - 1) / WG;
    const unsigned grid = (unsigned)(blocks < 4096 ? blocks : 4096);
    const uint64_t* fac = static_cast<const uint64_t*>(sp.d_factors.p);
    if (sp.tmpl == AT_TMPL_GEMM)
        hipLaunchKernelGGL(k_feature_scan<AT_TMPL_GEMM>, dim3(grid), dim3(WG), 0, stream, sd, fac, n, flags, ref);
    else
        hipLaunchKernelGGL(k_feature_scan<AT_TMPL_CONV2D_NCHW>, dim3(grid), dim3(WG), 0, stream, sd, fac, n, flags,
                           ref);
    return hipGetLastError();
}

hipError_t launch_export(const at_chains_s& ch, uint64_t* cur_cfg, float* cur_score, hipStream_t stream) {
    if (ch.n_chains == 0) return hipSuccess;
    const unsigned grid = (unsigned)((ch.n_chains + WG - 1) / WG);
    hipLaunchKernelGGL(k_export, dim3(grid), dim3(WG), 0, stream, static_cast<const SpaceDesc*>(ch.d_descs.p),
                       static_cast<const int64_t*>(ch.d_offsets.p), ch.n_spaces,
                       static_cast<const uint16_t*>(ch.d_knobs.p), static_cast<const float*>(ch.d_score.p),
                       ch.n_chains, cur_cfg, cur_score);
    return hipGetLastError();
}

}  // namespace at
