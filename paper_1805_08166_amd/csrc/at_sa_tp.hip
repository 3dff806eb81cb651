// Parallel simulated annealing (Section 3.3), tree-partitioned across the GPU.
//
// One annealing step of every chain is two kernels:
//   k_chain  one lane per chain: folds the leaf values of the candidate just
//            scored (tree order, fp32, from +0.0f), offers it to the chain's
//            best list, applies the Metropolis test, then proposes the next
//            candidate (one knob changed, Philox block (chain, step, 0, 0)),
//            evaluates its loop-context features and writes them as packed
//            bytes, quad-major (dword q of chain c at Fg[q * n + c]).
//   k_trees  workgroup w holds trees [w*tpw, (w+1)*tpw) in LDS and walks
//            them for every chain, 256 chains at a time through an LDS
//            feature tile, writing the reached leaf values to V.
// The kernel boundary is the only device-wide synchronisation: it is cheaper
// than an in-kernel grid barrier here because the cross-XCD data (features
// and leaf values) must be written back from the per-XCD L2 caches anyway.
//
// V is laid out in groups of four trees: the values of trees 4g..4g+3 for
// chain c are the 16 bytes at V[(g * n + c) * 4], so the fold reads one
// float4 per lane per group, coalesced across the wave.
#include "at_device.h"

namespace at {
namespace {

using namespace dev;

constexpr int TREE_WG = 256;
constexpr int CHAIN_WG = 256;           // one wave of chains + three loader waves
constexpr int CHAINS_PER_WG = 64;
constexpr int FOLD_GROUPS = 32;         // 4-tree groups per staged chunk (32 KB)
constexpr int LOAD_PER_THREAD = (FOLD_GROUPS * CHAINS_PER_WG + 191) / 192;
constexpr int TREE_LDS_BYTES = 65536;   // resident tree words per workgroup

enum { FIN_NONE = 0, FIN_INIT = 1, FIN_STEP = 2 };
enum { DRAW_NONE = 0, DRAW_INIT = 1, DRAW_PROPOSE = 2 };

struct ChainArgs {
    const SpaceDesc* descs;
    const int64_t* offsets;
    int n_spaces;
    const uint64_t* factors;
    uint16_t* knobs;          // [n][MAX_KNOBS] current configuration
    uint16_t* cand;           // [n][MAX_KNOBS] candidate being scored
    float* cur_score;         // [n]
    at_entry* top;            // [n][topk]
    ChainMeta* meta;          // [n]
    int topk;
    int64_t n;
    uint64_t chain0;
    uint64_t seed;
    const float* V;           // leaf values, groups of 4 trees
    int T;
    uint32_t* Fg;             // [Q][n] packed features
    int fin;                  // what the pending candidate is
    int fin_step;             // its local step index (thr / trace row)
    int steps;                // row length of thr and trace
    const float* thr;
    at_entry* trace;
    int draw;                 // what to propose next
    uint32_t draw_step;       // absolute step of the proposal
    at_entry* best;           // copy of the best lists (last launch), or null
};

__device__ __forceinline__ void load_knobs(const uint16_t* p, int64_t c, uint32_t (&kv)[MAX_KNOBS]) {
    const uint4 w = reinterpret_cast<const uint4*>(p)[c];
    const uint32_t pw[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) kv[j] = (pw[j >> 1] >> (16 * (j & 1))) & 0xffffu;
}

__device__ __forceinline__ void store_knobs(uint16_t* p, int64_t c, const uint32_t (&kv)[MAX_KNOBS]) {
    uint4 w;
    w.x = kv[0] | (kv[1] << 16);
    w.y = kv[2] | (kv[3] << 16);
    w.z = kv[4] | (kv[5] << 16);
    w.w = kv[6] | (kv[7] << 16);
    reinterpret_cast<uint4*>(p)[c] = w;
}

// Loads chunk k of the leaf values of this workgroup's chains into vbuf:
// element i is group (k * FOLD_GROUPS + i / 64), chain c0 + i % 64.  Called
// by the three loader waves; all loads are issued before the LDS stores.
__device__ __forceinline__ void load_fold_chunk(const float4* __restrict__ V4, int64_t n, int64_t c0, int nc,
                                                int groups, int k, float4* __restrict__ dst, int ltid) {
    float4 r[LOAD_PER_THREAD];
#pragma unroll
    for (int u = 0; u < LOAD_PER_THREAD; ++u) {
        const int i = ltid + u * 192;
        const int g = k * FOLD_GROUPS + i / CHAINS_PER_WG, j = i % CHAINS_PER_WG;
        r[u] = (i < FOLD_GROUPS * CHAINS_PER_WG && g < groups && j < nc) ? V4[(int64_t)g * n + c0 + j]
                                                                          : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < LOAD_PER_THREAD; ++u) {
        const int i = ltid + u * 192;
        if (i < FOLD_GROUPS * CHAINS_PER_WG) dst[i] = r[u];
    }
}

template <int TMPL>
__global__ __launch_bounds__(CHAIN_WG) void k_chain(ChainArgs a) {
    constexpr int A = (TMPL == AT_TMPL_GEMM) ? 3 : 6;
    constexpr int Q = (Nest<TMPL>::F + 3) / 4;
    __shared__ float4 vbuf[2][FOLD_GROUPS * CHAINS_PER_WG];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int64_t c0 = (int64_t)blockIdx.x * CHAINS_PER_WG;
    const int nc = (a.n - c0 < CHAINS_PER_WG) ? (int)(a.n - c0) : CHAINS_PER_WG;
    const int64_t c = c0 + (tid & 63);

    // score of the pending candidate: its leaves added in tree order.  The
    // leaf values are staged through LDS in chunks by waves 1-3 while wave 0
    // (one lane per chain) folds the previous chunk.
    float s = 0.0f;
    if (a.fin != FIN_NONE) {
        const float4* V4 = reinterpret_cast<const float4*>(a.V);
        const int groups = (a.T + 3) >> 2;
        const int chunks = (groups + FOLD_GROUPS - 1) / FOLD_GROUPS;
        if (wave > 0) load_fold_chunk(V4, a.n, c0, nc, groups, 0, vbuf[0], tid - 64);
        __syncthreads();
        for (int k = 0; k < chunks; ++k) {
            if (wave == 0) {
                const float4* src = vbuf[k & 1] + (tid & 63);
                const int g_end = (groups - k * FOLD_GROUPS < FOLD_GROUPS) ? groups - k * FOLD_GROUPS : FOLD_GROUPS;
#pragma unroll 8
                for (int g = 0; g < g_end; ++g) {
                    const float4 q = src[g * CHAINS_PER_WG];
                    const int t = (k * FOLD_GROUPS + g) * 4;
                    s = s + q.x;
                    if (t + 1 < a.T) s = s + q.y;
                    if (t + 2 < a.T) s = s + q.z;
                    if (t + 3 < a.T) s = s + q.w;
                }
            } else if (k + 1 < chunks) {
                load_fold_chunk(V4, a.n, c0, nc, groups, k + 1, vbuf[(k + 1) & 1], tid - 64);
            }
            __syncthreads();
        }
    }
    if (wave != 0 || (tid & 63) >= nc) return;

    int w = 0;
    while (w + 1 < a.n_spaces && a.offsets[w + 1] <= c) ++w;
    const SpaceDesc& sd = a.descs[w];
    const uint64_t gchain = a.chain0 + (uint64_t)c;
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    at_entry* list = a.top + c * a.topk;

    uint32_t cur[MAX_KNOBS];
    load_knobs(a.knobs, c, cur);

    if (a.fin != FIN_NONE) {
        uint32_t cd[MAX_KNOBS];
        load_knobs(a.cand, c, cd);
        uint64_t cfg = 0;
#pragma unroll
        for (int j = 0; j < MAX_KNOBS; ++j)
            if (j < sd.n_knobs) cfg += (uint64_t)cd[j] * sd.radix[j];
        ChainMeta m;
        if (a.fin == FIN_INIT) {
            for (int i = 0; i < a.topk; ++i) {
                at_entry z;
                z.cfg = 0;
                z.score = 0.0f;
                z.flag = 0u;
                list[i] = z;
            }
            m.count = 0;
            m.kth_score = 0.0f;
            m.kth_cfg = 0;
        } else {
            m = a.meta[c];
        }
        int count = (int)m.count;
        offer(list, a.topk, count, m.kth_score, m.kth_cfg, cfg, s);
        m.count = (uint32_t)count;
        a.meta[c] = m;
        bool acc;
        if (a.fin == FIN_INIT) {
            acc = true;
        } else {
            const float delta = s - a.cur_score[c];
            acc = delta >= a.thr[c * a.steps + a.fin_step];
            if (a.trace) {
                at_entry t;
                t.cfg = cfg;
                t.score = s;
                t.flag = acc ? 1u : 0u;
                a.trace[c * a.steps + a.fin_step] = t;
            }
        }
        if (acc) {
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j) cur[j] = cd[j];
            store_knobs(a.knobs, c, cur);
            a.cur_score[c] = s;
        }
    }

    if (a.draw != DRAW_NONE) {
        uint32_t cd[MAX_KNOBS];
        if (a.draw == DRAW_INIT) {
            // each knob uniform over its values: block (chain, 0, 1, j / 4)
            U4 r{0, 0, 0, 0};
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j) {
                if ((j & 3) == 0) r = philox(k0, k1, U4{(uint32_t)gchain, 0u, 1u, (uint32_t)(j >> 2)});
                const uint32_t word = (j & 3) == 0 ? r.x : (j & 3) == 1 ? r.y : (j & 3) == 2 ? r.z : r.w;
                cd[j] = (j < sd.n_knobs) ? uniform_below(word, sd.knob_size[j]) : 0u;
            }
        } else {
            const U4 r = philox(k0, k1, U4{(uint32_t)gchain, a.draw_step, 0u, 0u});
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j) cd[j] = cur[j];
            if (sd.n_mut > 0) {
                const int jm = sd.mut[uniform_below(r.x, (uint32_t)sd.n_mut)];
                uint32_t old = 0, size = 2;
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j)
                    if (j == jm) { old = cur[j]; size = sd.knob_size[j]; }
                uint32_t nv = uniform_below(r.y, size - 1u);
                if (nv >= old) nv += 1u;
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j)
                    if (j == jm) cd[j] = nv;
            }
        }
        store_knobs(a.cand, c, cd);
        uint32_t fac[6][4];
        gather_factors<TMPL>(sd, a.factors, cd, fac);
        uint32_t words[Q];
#pragma unroll
        for (int q = 0; q < Q; ++q) words[q] = 0u;
        nest_features<TMPL>(sd, fac, unroll_max_of(cd[A]), 1u + cd[A + 1],
                            [&](int f, uint32_t v) { words[f >> 2] |= v << (8 * (f & 3)); });
#pragma unroll
        for (int q = 0; q < Q; ++q) a.Fg[(int64_t)q * a.n + c] = words[q];
    }

    if (a.best) {
        for (int i = 0; i < a.topk; ++i) a.best[c * a.topk + i] = list[i];
    }
}

struct TreeArgs {
    EnsembleDesc e;
    const uint32_t* Fg;
    int64_t n;
    int Q;
    float* V;
    int tpw;              // trees per workgroup
};

template <int DEPTH, int GROUP>
__device__ __forceinline__ void walk_store(const uint32_t* __restrict__ trees, const uint8_t* __restrict__ tile_b,
                                           uint32_t fb, int t_local, int t_global, int64_t c, int64_t n,
                                           float* __restrict__ V, bool active) {
    constexpr int W = 2 << DEPTH;
    uint32_t lw[GROUP], li[GROUP];
    walk<DEPTH, GROUP>(trees, tile_b, fb, t_local * W, lw, li);
    if (active) {
#pragma unroll
        for (int g = 0; g < GROUP; ++g) {
            const int t = t_global + g;
            V[(((int64_t)(t >> 2) * n + c) << 2) + (t & 3)] = __uint_as_float(lw[g]);
        }
    }
}

// Walks `r` (< 2*H) trees starting at local tree t, in groups of H, H/2, ..., 1.
template <int DEPTH, int H>
__device__ __forceinline__ void walk_rest(const uint32_t* __restrict__ trees, const uint8_t* __restrict__ tile_b,
                                          uint32_t fb, int t, int t_global, int r, int64_t c, int64_t n,
                                          float* __restrict__ V, bool active) {
    if (r >= H) {
        walk_store<DEPTH, H>(trees, tile_b, fb, t, t_global, c, n, V, active);
        t += H;
        t_global += H;
        r -= H;
    }
    if constexpr (H > 1) walk_rest<DEPTH, H / 2>(trees, tile_b, fb, t, t_global, r, c, n, V, active);
}

template <int DEPTH, int Q>
__global__ __launch_bounds__(TREE_WG) void k_trees(TreeArgs a) {
    constexpr int W = 2 << DEPTH;
    constexpr int G = (DEPTH <= 8) ? 8 : 4;
    extern __shared__ uint32_t lds[];
    uint32_t* tile = lds;
    uint32_t* trees = lds + Q * TREE_WG;
    const uint8_t* tile_b = reinterpret_cast<const uint8_t*>(tile);
    const int tid = threadIdx.x;
    const int t0 = blockIdx.x * a.tpw;
    const int nt = (a.e.n_trees - t0 < a.tpw) ? (a.e.n_trees - t0) : a.tpw;
    if (nt <= 0) return;
    stage_words(trees, a.e.words + (size_t)t0 * W, nt * W);
    const uint32_t fb = tid * 4u;
    // the next block's features are fetched into registers during the walk
    uint32_t pre[Q];
#pragma unroll
    for (int q = 0; q < Q; ++q) pre[q] = (tid < a.n) ? a.Fg[(int64_t)q * a.n + tid] : 0u;
    for (int64_t cb = 0; cb < a.n; cb += TREE_WG) {
        __syncthreads();
#pragma unroll
        for (int q = 0; q < Q; ++q) tile[q * TREE_WG + tid] = pre[q];
        __syncthreads();
        const int64_t c = cb + tid;
        const bool active = c < a.n;
        const int64_t cn = c + TREE_WG;
        if (cb + TREE_WG < a.n) {
#pragma unroll
            for (int q = 0; q < Q; ++q) pre[q] = (cn < a.n) ? a.Fg[(int64_t)q * a.n + cn] : 0u;
        }
        int t = 0;
        for (; t + G <= nt; t += G) walk_store<DEPTH, G>(trees, tile_b, fb, t, t0 + t, c, a.n, a.V, active);
        walk_rest<DEPTH, G / 2>(trees, tile_b, fb, t, t0 + t, nt - t, c, a.n, a.V, active);
    }
}

template <int DEPTH, int Q>
hipError_t launch_trees_depth(const TreeArgs& a, hipStream_t stream) {
    constexpr int W = 2 << DEPTH;
    const size_t lds = (size_t)Q * TREE_WG * 4 + (size_t)a.tpw * W * 4;
    static bool configured = false;
    if (!configured) {
        hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_trees<DEPTH, Q>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             Q * TREE_WG * 4 + TREE_LDS_BYTES);
        if (err != hipSuccess) return err;
        configured = true;
    }
    const int grid = (a.e.n_trees + a.tpw - 1) / a.tpw;
    hipLaunchKernelGGL((k_trees<DEPTH, Q>), dim3(grid), dim3(TREE_WG), lds, stream, a);
    return hipGetLastError();
}

template <int Q>
hipError_t launch_trees_q(const TreeArgs& a, hipStream_t stream) {
    switch (a.e.depth) {
        case 1: return launch_trees_depth<1, Q>(a, stream);
        case 2: return launch_trees_depth<2, Q>(a, stream);
        case 3: return launch_trees_depth<3, Q>(a, stream);
        case 4: return launch_trees_depth<4, Q>(a, stream);
        case 5: return launch_trees_depth<5, Q>(a, stream);
        case 6: return launch_trees_depth<6, Q>(a, stream);
        case 7: return launch_trees_depth<7, Q>(a, stream);
        case 8: return launch_trees_depth<8, Q>(a, stream);
        case 9: return launch_trees_depth<9, Q>(a, stream);
        case 10: return launch_trees_depth<10, Q>(a, stream);
        case 11: return launch_trees_depth<11, Q>(a, stream);
        case 12: return launch_trees_depth<12, Q>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_trees(const TreeArgs& a, hipStream_t stream) {
    if (a.Q == 28) return launch_trees_q<28>(a, stream);   // GEMM: 110 features
    if (a.Q == 44) return launch_trees_q<44>(a, stream);   // conv2d: 176 features
    return hipErrorInvalidValue;
}

hipError_t ensure(DeviceBuf& b, size_t bytes) {
    if (b.p && b.bytes >= bytes) return hipSuccess;
    if (b.p) {
        hipError_t e = hipFree(b.p);
        if (e != hipSuccess) return e;
        b.p = nullptr;
        b.bytes = 0;
    }
    hipError_t e = hipMalloc(&b.p, bytes);
    if (e != hipSuccess) {
        b.p = nullptr;
        return e;
    }
    b.bytes = bytes;
    return hipSuccess;
}

}  // namespace

hipError_t launch_sa_tp(const at_space_s& sp, const EnsembleDesc& e, at_chains_s& ch, int steps, bool init,
                        const float* thr, at_entry* best, at_entry* trace, hipStream_t stream) {
    const int64_t n = ch.n_chains;
    if (n == 0) return hipSuccess;
    const int Q = (sp.descs[0].n_features + 3) / 4;
    const int groups = (e.n_trees + 3) / 4;
    hipError_t err;
    if ((err = ensure(ch.d_cand, (size_t)n * MAX_KNOBS * 2)) != hipSuccess) return err;
    if ((err = ensure(ch.d_meta, (size_t)n * sizeof(ChainMeta))) != hipSuccess) return err;
    if ((err = ensure(ch.d_fg, (size_t)Q * n * 4)) != hipSuccess) return err;
    if ((err = ensure(ch.d_v, (size_t)groups * n * 16)) != hipSuccess) return err;

    ChainArgs ca{};
    ca.descs = static_cast<const SpaceDesc*>(sp.d_descs.p);
    ca.offsets = static_cast<const int64_t*>(sp.d_offsets.p);
    ca.n_spaces = sp.n_spaces;
    ca.factors = static_cast<const uint64_t*>(sp.d_factors.p);
    ca.knobs = static_cast<uint16_t*>(ch.d_knobs.p);
    ca.cand = static_cast<uint16_t*>(ch.d_cand.p);
    ca.cur_score = static_cast<float*>(ch.d_score.p);
    ca.top = static_cast<at_entry*>(ch.d_top.p);
    ca.meta = static_cast<ChainMeta*>(ch.d_meta.p);
    ca.topk = ch.topk;
    ca.n = n;
    ca.chain0 = (uint64_t)ch.chain0;
    ca.seed = ch.seed;
    ca.V = static_cast<const float*>(ch.d_v.p);
    ca.T = e.n_trees;
    ca.Fg = static_cast<uint32_t*>(ch.d_fg.p);
    ca.steps = steps;
    ca.thr = thr;
    ca.trace = trace;

    TreeArgs ta{};
    ta.e = e;
    ta.Fg = ca.Fg;
    ta.n = n;
    ta.Q = Q;
    ta.V = static_cast<float*>(ch.d_v.p);
    // spread the trees over the compute units, within the LDS budget
    int n_cu = 256;
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, ch.device);
    const int W = 2 << e.depth;
    int tpw = (e.n_trees + n_cu - 1) / n_cu;
    const int tpw_max = TREE_LDS_BYTES / (W * 4) > 0 ? TREE_LDS_BYTES / (W * 4) : 1;
    if (tpw > tpw_max) tpw = tpw_max;
    if (tpw < 1) tpw = 1;
    ta.tpw = tpw;

    const unsigned chain_grid = (unsigned)((n + CHAINS_PER_WG - 1) / CHAINS_PER_WG);
    auto chain_kernel = [&](const ChainArgs& x) -> hipError_t {
        if (sp.tmpl == AT_TMPL_GEMM)
            hipLaunchKernelGGL(k_chain<AT_TMPL_GEMM>, dim3(chain_grid), dim3(CHAIN_WG), 0, stream, x);
        else
            hipLaunchKernelGGL(k_chain<AT_TMPL_CONV2D_NCHW>, dim3(chain_grid), dim3(CHAIN_WG), 0, stream, x);
        return hipGetLastError();
    };

    int pending = FIN_NONE;
    if (init) {
        ChainArgs x = ca;
        x.fin = FIN_NONE;
        x.draw = DRAW_INIT;
        if ((err = chain_kernel(x)) != hipSuccess) return err;
        if ((err = launch_trees(ta, stream)) != hipSuccess) return err;
        pending = FIN_INIT;
    }
    for (int s = 0; s < steps; ++s) {
        ChainArgs x = ca;
        x.fin = pending;
        x.fin_step = s - 1;
        x.draw = DRAW_PROPOSE;
        x.draw_step = (uint32_t)(ch.step_abs + (uint64_t)s);
        if ((err = chain_kernel(x)) != hipSuccess) return err;
        if ((err = launch_trees(ta, stream)) != hipSuccess) return err;
        pending = FIN_STEP;
    }
    ChainArgs x = ca;
    x.fin = pending;
    x.fin_step = steps - 1;
    x.draw = DRAW_NONE;
    x.best = best;
    return chain_kernel(x);
}

}  // namespace at
