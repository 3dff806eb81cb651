// Parallel simulated annealing (Section 3.3), chain-local.
//
// One persistent workgroup owns `cpb` chains for the whole run: every
// scoring round (the initial draw, then one round per annealing step) it
// proposes, featurises, scores, offers and accepts without leaving the
// kernel, so a run is one launch.  The ensemble does not fit one compute
// unit's LDS, so each round streams it through a two-buffer LDS ring in
// chunks of `ct` trees (direct global-to-LDS loads, 16 bytes per lane);
// it stays resident in the per-XCD L2 across rounds.  When the whole
// ensemble fits, it is loaded once.
//
// Waves: wave 0 folds leaf values (one lane per chain, fp32 from +0.0f in
// tree order, one chunk behind the walk) and runs the per-chain bookkeeping;
// waves 1.. walk the trees.  A walk lane handles chain (lane % cpb) and up
// to four trees at a time.  The candidates' features sit in a 64-column
// tile at LDS offset 0 (byte (f & 3) of dword (f >> 2) * 64 + column holds
// 4x+3, column l for chain l % cpb), so the walk's feature address is one
// and-or of the node and the lane's column.
//
// Tree layout in the ring ("local form"): tree t occupies `ts` words, the
// compact node block (2^(d-1) words) followed, when leaves are streamed, by
// the 2^d leaf values; ts is odd, so the same node word of consecutive
// trees falls in consecutive LDS banks.  With `gather` set only node
// blocks are streamed and each walk reads its one leaf from global memory.
#include <hip/hip_ext.h>

#include "at_chain.h"

namespace at {
namespace {

using namespace dev;

constexpr int LOCAL_WG_MAX = 512;
constexpr int LOCAL_FAC_MAX = 1024;          // split choices staged in LDS
constexpr uint32_t LOCAL_TILE_MASK = 0x3f03u;  // node bits of a tile byte address (tile below 16 KB)
// dynamic LDS per workgroup: the compute unit's 160 KB less 1 KB kept for
// any static LDS the compiler places
constexpr size_t LOCAL_LDS_BYTES = 163840 - 1024;

struct LocalArgs {
    const SpaceDesc* descs;
    const int64_t* offsets;
    int n_spaces;
    const uint64_t* factors;
    uint16_t* knobs;          // [n][MAX_KNOBS] current configuration
    float* cur_score;         // [n]
    at_entry* top;            // [n][topk] best lists
    ChainMeta* meta;          // [n]
    int topk;
    int cpb;                  // chains per workgroup (a divisor of 64)
    int64_t n;
    uint64_t chain0;
    uint64_t seed;
    int init;                 // first round draws, scores and offers the initial configurations
    int steps;
    uint32_t step0;           // absolute step of local step 0
    const float* thr;         // [n][steps]
    at_entry* trace;          // [n][steps] or null
    at_entry* best;           // [n][topk]
    const uint32_t* tw;       // local form, tree t at words [t * ts, (t + 1) * ts)
    int ts;
    int T;
    int ct;                   // trees per chunk, a multiple of 4 and at most 4 per walk slot
    int n_chunks;
    int resident;             // the ring holds every tree (loaded once); else two chunk buffers
    int gather;               // leaves from global memory (leaf_src) instead of the ring
    const uint32_t* leaf_src; // compact form: leaves of tree t at leaf_src[t * w16 + 2^(d-1) + q]
    int w16;
    // dynamic LDS layout (byte offsets; the feature tile is at 0)
    uint32_t off_ring, ring_bytes;
    uint32_t off_lv;
    int lv_stride;            // floats per chain row of leaf values: two chunk slots (one when resident)
    uint32_t off_lists, off_rec, off_frow, off_desc;
};

// Leaf indices of four trees for this lane: nb holds the LDS byte offsets
// of the trees' node blocks (per lane), fb the lane's tile column.  The
// levels are those of the tree kernel's walk (five vector instructions per
// level and tree); trees are independent, so their LDS round trips overlap.
template <int DEPTH>
__device__ __forceinline__ void walk4_local(const uint8_t* __restrict__ L, const uint32_t (&nb)[4], uint32_t fb,
                                            uint32_t (&q)[4]) {
    uint32_t node[4], p[4], fa[4], pa[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        node[g] = *reinterpret_cast<const uint16_t*>(L + nb[g]);
        p[g] = 1u;
        fa[g] = (node[g] & LOCAL_TILE_MASK) | fb;
        pa[g] = nb[g] + 4u;
    }
#pragma unroll
    for (int l = 0; l + 1 < DEPTH; ++l) {
        uint32_t x4[4], pr[4];
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            x4[g] = L[fa[g]];
            pr[g] = *reinterpret_cast<const uint32_t*>(L + pa[g]);
        }
        const uint32_t mask = LOCAL_TILE_MASK;
        asm(AT_WALK4_ASM
            : "+v"(node[0]), "+v"(node[1]), "+v"(node[2]), "+v"(node[3]), "+v"(p[0]), "+v"(p[1]), "+v"(p[2]),
              "+v"(p[3]), "=&v"(fa[0]), "=&v"(fa[1]), "=&v"(fa[2]), "=&v"(fa[3]), "=&v"(pa[0]), "=&v"(pa[1]),
              "=&v"(pa[2]), "=&v"(pa[3])
            : "v"(x4[0]), "v"(x4[1]), "v"(x4[2]), "v"(x4[3]), "v"(pr[0]), "v"(pr[1]), "v"(pr[2]), "v"(pr[3]),
              "s"(mask), "v"(fb), "v"(nb[0]), "v"(nb[1]), "v"(nb[2]), "v"(nb[3])
            : "vcc");
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const uint32_t x4 = L[fa[g]];
        q[g] = 2u * p[g] + (x4 >= (node[g] & 0xffu) ? 1u : 0u) - (1u << DEPTH);
    }
}

// Issues the direct-to-LDS loads of trees [t0, t0 + nt) of the local form
// into LDS at dst (one wave, 16 bytes per lane and instruction).
__device__ __forceinline__ void load_trees(const LocalArgs& a, uint8_t* dst, int t0, int nt, int lane) {
    const int n16 = (nt * a.ts * 4 + 15) >> 4;
    const uint4* src = reinterpret_cast<const uint4*>(a.tw + (size_t)t0 * a.ts);
    uint4* d = reinterpret_cast<uint4*>(dst);
    for (int base = 0; base < n16; base += 64) {
        const int i = base + lane;
        if (i < n16) __builtin_amdgcn_global_load_lds(src + i, d + base, 16, 0, 0);
    }
}

// Workgroup barrier that orders LDS accesses only: each wave's own LDS
// operations complete before it arrives; global loads stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int TMPL, int DEPTH>
__global__ __launch_bounds__(LOCAL_WG_MAX) void k_local(LocalArgs a) {
    using N = Nest<TMPL>;
    constexpr int A = (TMPL == AT_TMPL_GEMM) ? 3 : 6;
    constexpr int Q = (N::F + 3) / 4;
    constexpr int RS = Q * 4 + 4;
    constexpr uint32_t NBB = 4u << (DEPTH - 1);   // node block bytes
    extern __shared__ uint4 lds4[];
    uint8_t* lds = reinterpret_cast<uint8_t*>(lds4);
    uint32_t* tile = reinterpret_cast<uint32_t*>(lds);
    uint8_t* ring = lds + a.off_ring;
    float* lv = reinterpret_cast<float*>(lds + a.off_lv);
    at_entry* lists = reinterpret_cast<at_entry*>(lds + a.off_lists);
    ChainRec* rec = reinterpret_cast<ChainRec*>(lds + a.off_rec);
    uint8_t* frow = lds + a.off_frow;
    SpaceDesc& s_desc = *reinterpret_cast<SpaceDesc*>(lds + a.off_desc);
    uint64_t* s_fac = reinterpret_cast<uint64_t*>(lds + a.off_desc + sizeof(SpaceDesc));

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nthreads = (int)blockDim.x;
    const int cpb = a.cpb;
    const int64_t c0 = (int64_t)blockIdx.x * cpb;
    const int nc = (a.n - c0 < cpb) ? (int)(a.n - c0) : cpb;
    const int k = a.topk;
    const bool owner = tid < nc;
    const int64_t c = c0 + (owner ? tid : 0);
    const int gj = tid >> 4, gr = tid & 15;
    const uint64_t gmask = 0xffffull << (16 * (gj & 3));
    const bool gvalid = gj < nc;
    const int gjc = gvalid ? gj : 0;

    // space tables: staged in LDS when every chain of the workgroup uses one space
    const int w_lo = space_of(a.offsets, a.n_spaces, c0), w_hi = space_of(a.offsets, a.n_spaces, c0 + nc - 1);
    int fac_lo = 0, fac_n = 0;
    if (w_lo == w_hi) {
        const SpaceDesc& g = a.descs[w_lo];
        fac_lo = g.split_off[0];
        for (int ax = 0; ax < g.n_axes; ++ax) fac_n += (int)g.knob_size[ax];
    }
    const bool staged = w_lo == w_hi && fac_n <= LOCAL_FAC_MAX;
    if (staged) {
        constexpr int DW = (int)(sizeof(SpaceDesc) / 4);
        constexpr int SO = (int)(offsetof(SpaceDesc, split_off) / 4);
        const uint32_t* gd = reinterpret_cast<const uint32_t*>(a.descs + w_lo);
        uint32_t* ld = reinterpret_cast<uint32_t*>(&s_desc);
        for (int i = tid; i < DW; i += nthreads)
            ld[i] = (i >= SO && i < SO + MAX_AXES) ? gd[i] - (uint32_t)fac_lo : gd[i];
        for (int i = tid; i < fac_n; i += nthreads) s_fac[i] = a.factors[fac_lo + i];
    }
    const uint64_t* facp = staged ? s_fac : a.factors;
    const SpaceDesc* sdp = staged ? &s_desc : a.descs + space_of(a.offsets, a.n_spaces, c);
    const SpaceDesc* gsdp = staged ? &s_desc : a.descs + space_of(a.offsets, a.n_spaces, c0 + gjc);

    // chain state: knobs and score in the owner lanes, best lists and their
    // bookkeeping in LDS
    uint32_t cur[MAX_KNOBS];
    float cur_s = 0.0f;
    if (owner) {
        load_knobs(a.knobs, c, cur);
        cur_s = a.cur_score[c];
        ChainRec& R = rec[tid];
        if (a.init) {
            R.count = 0;
            R.kth_score = 0.0f;
            R.kth_cfg = 0;
        } else {
            const ChainMeta m = a.meta[c];
            R.count = m.count;
            R.kth_score = m.kth_score;
            R.kth_cfg = m.kth_cfg;
        }
    }
    for (int e = tid; e < nc * k; e += nthreads) {
        if (a.init) {
            at_entry z;
            z.cfg = 0;
            z.score = 0.0f;
            z.flag = 0u;
            lists[e] = z;
        } else {
            lists[e] = a.top[c0 * k + e];
        }
    }

    // the staged tables, initial lists and records are in place
    lds_barrier();
    const int rounds = (a.init ? 1 : 0) + a.steps;
    const bool resident = a.resident != 0;
    const int nck = a.n_chunks;
    const int total_chunks = rounds * nck;
    // the loader wave starts the first chunk (the whole ensemble when resident)
    if (wave == 1 && rounds > 0) {
        if (resident) load_trees(a, ring, 0, a.T, lane);
        else load_trees(a, ring, 0, a.ct < a.T ? a.ct : a.T, lane);
    }

    // walk-lane geometry: chain jw, tree slot u of S (four trees per lane and chunk)
    const int wt = tid - 128;                     // walk thread (waves 2..)
    const int jw = lane % cpb;
    const int S = (nthreads - 128) / cpb;
    const int u = (wt >= 0 ? wt : 0) / cpb;
    const uint32_t fb = (uint32_t)lane * 4u;
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    const uint64_t gchain = a.chain0 + (uint64_t)c;
    // threshold of the owner's next step, loaded one round ahead
    float thr_next = (owner && a.steps > 0) ? a.thr[c * a.steps] : 0.0f;

    for (int r = 0; r < rounds; ++r) {
        const bool is_init = a.init && r == 0;
        const int s = r - (a.init ? 1 : 0);
        // (1) candidate: the initial draw (block (chain, 0, 1, j / 4)) or one
        // knob moved to another value (block (chain, step, 0, 0))
        uint32_t cd[MAX_KNOBS];
        float thr_v = 0.0f;
        if (owner) {
            const SpaceDesc& sd = *sdp;
            if (is_init) {
                U4 rr{0, 0, 0, 0};
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j) {
                    if ((j & 3) == 0) rr = philox(k0, k1, U4{(uint32_t)gchain, 0u, 1u, (uint32_t)(j >> 2)});
                    const uint32_t word = (j & 3) == 0 ? rr.x : (j & 3) == 1 ? rr.y : (j & 3) == 2 ? rr.z : rr.w;
                    cd[j] = (j < sd.n_knobs) ? uniform_below(word, sd.knob_size[j]) : 0u;
                }
            } else {
                thr_v = thr_next;
                if (s + 1 < a.steps) thr_next = a.thr[c * a.steps + s + 1];
                const U4 rr = philox(k0, k1, U4{(uint32_t)gchain, a.step0 + (uint32_t)s, 0u, 0u});
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j) cd[j] = cur[j];
                if (sd.n_mut > 0) {
                    const int jm = sd.mut[uniform_below(rr.x, (uint32_t)sd.n_mut)];
                    uint32_t old = 0, size = 2;
#pragma unroll
                    for (int j = 0; j < MAX_KNOBS; ++j)
                        if (j == jm) { old = cur[j]; size = sd.knob_size[j]; }
                    uint32_t nv = uniform_below(rr.y, size - 1u);
                    if (nv >= old) nv += 1u;
#pragma unroll
                    for (int j = 0; j < MAX_KNOBS; ++j)
                        if (j == jm) cd[j] = nv;
                }
            }
#pragma unroll
            for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].nx[j] = cd[2 * j] | (cd[2 * j + 1] << 16);
        }
        lds_barrier();
        // (2) features: lane gr of group gj evaluates loop gr of chain gj
        if (gvalid && gr < N::L) {
            const SpaceDesc& sd = *gsdp;
            uint32_t nx[MAX_KNOBS];
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j) nx[j] = (rec[gj].nx[j >> 1] >> (16 * (j & 1))) & 0xffffu;
            uint32_t fac[6][4];
            gather_factors<TMPL>(sd, facp, nx, fac);
            uint32_t f[11];
            loop_features<TMPL>(sd, fac, unroll_max_of(nx[A]), 1u + nx[A + 1], gr, f);
#pragma unroll
            for (int i = 0; i < 11; ++i) frow[gj * RS + gr * 11 + i] = (uint8_t)f[i];
        }
        lds_barrier();
        // (3) the tile: column l holds chain l % cpb (the last chain stands
        // in for missing ones), bytes 4x+3
        for (int i = tid; i < Q * 64; i += nthreads) {
            const int q = i >> 6;
            int j = (i & 63) % cpb;
            j = j < nc ? j : nc - 1;
            uint32_t w = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int f = 4 * q + b;
                if (f < N::F) w |= (4u * frow[j * RS + f] + 3u) << (8 * b);
            }
            tile[i] = w;
        }
        // (4) chunk pipeline.  Iteration it: the loader brings the next chunk;
        // walkers walk chunk it, write the leaf values of chunk it - 1 (held
        // in registers since the last iteration) and fetch those of chunk it;
        // the fold wave adds chunk it - 2.
        float sc = 0.0f;
        uint32_t vprev[4] = {0u, 0u, 0u, 0u};
        int tprev[4] = {-1, -1, -1, -1};
        for (int it = 0; it <= nck; ++it) {
            const int gc = r * nck + it;
            if (wave == 1 && it < nck) __builtin_amdgcn_s_waitcnt(0);   // chunk it has landed
            lds_barrier();
            if (wave == 1) {
                if (!resident && it < nck && gc + 1 < total_chunks) {
                    const int x = (it + 1) % nck;
                    const int t0 = x * a.ct;
                    load_trees(a, ring + (size_t)((gc + 1) & 1) * a.ring_bytes, t0,
                               (a.T - t0 < a.ct ? a.T - t0 : a.ct), lane);
                }
            } else if (wave >= 2) {
                uint32_t q[4];
                int ti[4] = {-1, -1, -1, -1};
                const int t0 = it * a.ct;
                const int nt = it < nck ? (a.T - t0 < a.ct ? a.T - t0 : a.ct) : 0;
                uint32_t nb[4];
                if (nt > 0) {
                    // chunk it: resident trees sit at their own place, streamed
                    // ones in buffer gc & 1
                    const uint32_t rb = a.off_ring + (resident ? (uint32_t)t0 * (uint32_t)a.ts * 4u
                                                               : (uint32_t)(gc & 1) * a.ring_bytes);
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int tl = u + g * S;
                        ti[g] = tl < nt ? tl : -1;
                        nb[g] = rb + (uint32_t)(tl < nt ? tl : 0) * (uint32_t)a.ts * 4u;
                    }
                    walk4_local<DEPTH>(lds, nb, fb, q);
                }
                if (it > 0 && jw < nc) {
                    float* lvk = lv + ((it - 1) & 1) * a.ct + jw * a.lv_stride;
#pragma unroll
                    for (int g = 0; g < 4; ++g)
                        if (tprev[g] >= 0) lvk[tprev[g]] = __uint_as_float(vprev[g]);
                }
                if (nt > 0) {
                    if (a.gather) {
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int tt = ti[g] >= 0 ? ti[g] : 0;
                            vprev[g] = a.leaf_src[(size_t)(t0 + tt) * a.w16 + (NBB / 4) + q[g]];
                        }
                    } else {
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            vprev[g] = *reinterpret_cast<const uint32_t*>(lds + nb[g] + NBB + 4u * q[g]);
                    }
                }
#pragma unroll
                for (int g = 0; g < 4; ++g) tprev[g] = ti[g];
            } else if (it >= 2 && lane < nc) {
                // fold chunk it - 2 (a whole one), in tree order
                const float* row = lv + lane * a.lv_stride + (it & 1) * a.ct;
                for (int t = 0; t < a.ct; t += 4) {
                    const float4 v4 = *reinterpret_cast<const float4*>(row + t);
                    sc = sc + v4.x;
                    sc = sc + v4.y;
                    sc = sc + v4.z;
                    sc = sc + v4.w;
                }
            }
        }
        // the last chunk's leaf values are in place
        lds_barrier();
        if (wave == 0 && lane < nc) {
            const int last = nck - 1;
            const float* row = lv + lane * a.lv_stride + (last & 1) * a.ct;
            const int nt = a.T - last * a.ct;
            int t = 0;
            for (; t + 4 <= nt; t += 4) {
                const float4 v4 = *reinterpret_cast<const float4*>(row + t);
                sc = sc + v4.x;
                sc = sc + v4.y;
                sc = sc + v4.z;
                sc = sc + v4.w;
            }
            for (; t < nt; ++t) sc = sc + row[t];
        }
        // (5) offer to the best list, then the Metropolis test
        uint64_t cfg = 0;
        if (owner) {
            const SpaceDesc& sd = *sdp;
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j)
                if (j < sd.n_knobs) cfg += (uint64_t)cd[j] * sd.radix[j];
            ChainRec& R = rec[tid];
            const bool qual = is_init || (int)R.count < k || precedes(sc, cfg, R.kth_score, R.kth_cfg);
            R.cfg = cfg;
            R.score = sc;
            R.qual = qual ? 1u : 0u;
        }
        lds_barrier();
        if (gj < cpb) group_offer(lists + gjc * k, rec[gjc], k, gr, gmask, gvalid && rec[gjc].qual != 0);
        lds_barrier();
        if (owner) {
            bool acc = true;
            if (!is_init) {
                acc = (sc - cur_s) >= thr_v;
                if (a.trace) {
                    at_entry tr;
                    tr.cfg = cfg;
                    tr.score = sc;
                    tr.flag = acc ? 1u : 0u;
                    a.trace[c * a.steps + s] = tr;
                }
            }
            if (acc) {
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j) cur[j] = cd[j];
                cur_s = sc;
            }
        }
    }

    // write the chain state and the best lists back
    __syncthreads();
    if (owner) {
        store_knobs(a.knobs, c, cur);
        a.cur_score[c] = cur_s;
        ChainMeta m;
        m.count = rec[tid].count;
        m.kth_score = rec[tid].kth_score;
        m.kth_cfg = rec[tid].kth_cfg;
        a.meta[c] = m;
    }
    for (int e = tid; e < nc * k; e += nthreads) {
        const at_entry x = lists[e];
        a.top[c0 * k + e] = x;
        a.best[c0 * k + e] = x;
    }
}

template <int TMPL>
hipError_t launch_local_t(const LocalArgs& a, int depth, int grid, int threads, size_t lds, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop) {
    const void* fn = nullptr;
    switch (depth) {
#define AT_LOCAL_CASE(D) \
    case D: fn = reinterpret_cast<const void*>(&k_local<TMPL, D>); break;
        AT_LOCAL_CASE(1) AT_LOCAL_CASE(2) AT_LOCAL_CASE(3) AT_LOCAL_CASE(4) AT_LOCAL_CASE(5) AT_LOCAL_CASE(6)
        AT_LOCAL_CASE(7) AT_LOCAL_CASE(8) AT_LOCAL_CASE(9) AT_LOCAL_CASE(10) AT_LOCAL_CASE(11) AT_LOCAL_CASE(12)
#undef AT_LOCAL_CASE
        default: return hipErrorInvalidValue;
    }
    static bool configured[13] = {};
    if (!configured[depth]) {
        hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)LOCAL_LDS_BYTES);
        if (e != hipSuccess) return e;
        configured[depth] = true;
    }
    void* args[] = {const_cast<LocalArgs*>(&a)};
    if (start) {
        hipError_t e = hipEventRecord(start, stream);
        if (e != hipSuccess) return e;
    }
    hipError_t e = hipLaunchKernel(fn, dim3(grid), dim3(threads), args, lds, stream);
    if (e != hipSuccess) return e;
    if (stop) return hipEventRecord(stop, stream);
    return hipSuccess;
}

}  // namespace

// Smallest word stride >= words that is 1 mod 32.
int local_tree_stride(int words) { return words + ((1 - words) % 32 + 32) % 32; }

// Plan of the chain-local path for a run, or false when it does not fit.
// Workgroups of 512 threads: wave 0 folds and keeps the books, wave 1 loads
// trees, waves 2-7 walk.  Chains per workgroup: the smallest divisor of 64
// that leaves at most one workgroup per compute unit (at most 32).  A chunk
// holds at most four trees per walk slot.
bool plan_local(const at_space_s& sp, const EnsembleDesc& e, const at_chains_s& ch, LocalPlan& pl) {
    const int64_t n = ch.n_chains;
    const int Q = (sp.descs[0].n_features + 3) / 4;
    const int d = e.depth;
    const int NB = 1 << (d - 1), NL = 1 << d;
    const int T = e.n_trees;
    int n_cu = 256;
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, ch.device);
    int cpb = 1;
    while (cpb < 32 && (n + cpb - 1) / cpb > n_cu) cpb *= 2;
    const int threads = 512;
    const int slots = (threads - 128) / cpb;
    const int ct_cap = 4 * slots / 4 * 4;
    int fac_max = 0;
    for (const SpaceDesc& x : sp.descs) {
        int f = 0;
        for (int ax = 0; ax < x.n_axes; ++ax) f += (int)x.knob_size[ax];
        fac_max = f > fac_max ? f : fac_max;
    }
    if (fac_max > LOCAL_FAC_MAX) fac_max = LOCAL_FAC_MAX;
    const int RS = Q * 4 + 4;
    auto al16 = [](size_t x) { return (x + 15) & ~(size_t)15; };
    const size_t tile = (size_t)Q * 256;
    const size_t fixed = al16((size_t)cpb * ch.topk * sizeof(at_entry)) + al16((size_t)cpb * sizeof(ChainRec)) +
                         al16((size_t)cpb * RS) + al16(sizeof(SpaceDesc) + (size_t)fac_max * 8);
    if (tile + fixed >= LOCAL_LDS_BYTES) return false;
    const size_t avail = LOCAL_LDS_BYTES - tile - fixed;
    const int ts_full = local_tree_stride(NB + NL), ts_nodes = local_tree_stride(NB);
    auto lv_bytes = [&](int ct) { return al16((size_t)cpb * (2 * (size_t)ct + 4) * 4); };
    pl = LocalPlan{};
    pl.cpb = cpb;
    pl.threads = threads;
    pl.grid = (int)((n + cpb - 1) / cpb);
    pl.off_ring = (uint32_t)tile;
    // resident: every tree in LDS, loaded once, walked in chunks of ct
    const int ct_res = T <= ct_cap ? T : ct_cap;
    const size_t res_bytes = al16((size_t)T * ts_full * 4);
    if (res_bytes + lv_bytes(ct_res) <= avail) {
        pl.resident = 1;
        pl.gather = 0;
        pl.ts = ts_full;
        pl.ct = ct_res;
        pl.ring_bytes = (uint32_t)res_bytes;
    } else {
        // streamed in chunks through two buffers.  Leaves are gathered from
        // global memory when that moves fewer bytes per round than streaming
        // them (a 64-byte line per chain and tree against the leaf block).
        const double stream_full = (double)T * ts_full * 4;
        const double stream_nodes = (double)T * ts_nodes * 4 + (double)cpb * T * 64;
        pl.resident = 0;
        pl.gather = stream_nodes < stream_full ? 1 : 0;
        pl.ts = pl.gather ? ts_nodes : ts_full;
        // per tree of a chunk: two ring copies and two leaf-value slots per chain
        const size_t per_tree = 8 * ((size_t)pl.ts + cpb);
        const size_t spare = avail > (size_t)cpb * 16 + 64 ? avail - (size_t)cpb * 16 - 64 : 0;
        int ct_max = (int)(spare / per_tree) / 4 * 4;
        ct_max = ct_max < ct_cap ? ct_max : ct_cap;
        if (ct_max < 4) return false;
        const int chunks = (T + ct_max - 1) / ct_max;
        pl.ct = ((T + chunks - 1) / chunks + 3) / 4 * 4;
        pl.ring_bytes = (uint32_t)al16((size_t)pl.ct * pl.ts * 4);
    }
    pl.n_chunks = (T + pl.ct - 1) / pl.ct;
    pl.lv_stride = 2 * pl.ct + 4;
    size_t off = tile + (pl.resident ? 1 : 2) * (size_t)pl.ring_bytes;
    pl.off_lv = (uint32_t)off;
    off += lv_bytes(pl.ct);
    pl.off_lists = (uint32_t)off;
    off += al16((size_t)cpb * ch.topk * sizeof(at_entry));
    pl.off_rec = (uint32_t)off;
    off += al16((size_t)cpb * sizeof(ChainRec));
    pl.off_frow = (uint32_t)off;
    off += al16((size_t)cpb * RS);
    pl.off_desc = (uint32_t)off;
    off += al16(sizeof(SpaceDesc) + (size_t)fac_max * 8);
    pl.lds_bytes = off;
    // streamed bytes per round and workgroup, for the path choice
    pl.round_bytes = pl.resident ? 0.0 : (double)T * pl.ts * 4 + (pl.gather ? (double)cpb * T * 64 : 0.0);
    return pl.lds_bytes <= LOCAL_LDS_BYTES;
}

hipError_t launch_sa_local(const at_space_s& sp, const EnsembleDesc& e, at_chains_s& ch, const LocalPlan& pl,
                           int steps, bool init, const float* thr, at_entry* best, at_entry* trace,
                           hipStream_t stream) {
    const int64_t n = ch.n_chains;
    if (n == 0) return hipSuccess;
    hipError_t err;
    if (!ch.d_meta.p) {
        err = hipMalloc(&ch.d_meta.p, (size_t)n * sizeof(ChainMeta));
        if (err != hipSuccess) {
            ch.d_meta.p = nullptr;
            return err;
        }
        ch.d_meta.bytes = (size_t)n * sizeof(ChainMeta);
    }
    LocalArgs a{};
    a.descs = static_cast<const SpaceDesc*>(sp.d_descs.p);
    a.offsets = static_cast<const int64_t*>(sp.d_offsets.p);
    a.n_spaces = sp.n_spaces;
    a.factors = static_cast<const uint64_t*>(sp.d_factors.p);
    a.knobs = static_cast<uint16_t*>(ch.d_knobs.p);
    a.cur_score = static_cast<float*>(ch.d_score.p);
    a.top = static_cast<at_entry*>(ch.d_top.p);
    a.meta = static_cast<ChainMeta*>(ch.d_meta.p);
    a.topk = ch.topk;
    a.cpb = pl.cpb;
    a.n = n;
    a.chain0 = (uint64_t)ch.chain0;
    a.seed = ch.seed;
    a.init = init ? 1 : 0;
    a.steps = steps;
    a.step0 = (uint32_t)ch.step_abs;
    a.thr = thr;
    a.trace = trace;
    a.best = best;
    a.tw = pl.gather ? e.local_nodes : e.local_full;
    a.ts = pl.ts;
    a.T = e.n_trees;
    a.ct = pl.ct;
    a.n_chunks = pl.n_chunks;
    a.resident = pl.resident;
    a.gather = pl.gather;
    a.leaf_src = e.words16;
    a.w16 = 3 << (e.depth - 1);
    a.off_ring = pl.off_ring;
    a.ring_bytes = pl.ring_bytes;
    a.off_lv = pl.off_lv;
    a.lv_stride = pl.lv_stride;
    a.off_lists = pl.off_lists;
    a.off_rec = pl.off_rec;
    a.off_frow = pl.off_frow;
    a.off_desc = pl.off_desc;
    ch.events_used[0] = ch.events_used[1] = 0;
    hipEvent_t start = nullptr, stop = nullptr;
    if ((err = next_events(ch, 0, start, stop)) != hipSuccess) return err;
    if (sp.tmpl == AT_TMPL_GEMM)
        return launch_local_t<AT_TMPL_GEMM>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream, start, stop);
    return launch_local_t<AT_TMPL_CONV2D_NCHW>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream, start, stop);
}

}  // namespace at
