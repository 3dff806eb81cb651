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
    int walk_waves;           // waves 1 .. walk_waves walk; later waves load
    int tail;                 // tops resident (local_top), last level and leaves from the tail records
    const uint4* tail_rec;    // [T][2^(d-1)] records {node, left leaf, right leaf, 0}
    int gather;               // leaves from global memory (leaf_src) instead of the ring
    const uint32_t* leaf_src; // compact form: leaves of tree t at leaf_src[t * w16 + 2^(d-1) + q]
    int w16;
    // dynamic LDS layout (byte offsets; the feature tile is at 0)
    uint32_t off_ring, ring_bytes;
    uint32_t off_lv;
    int lv_stride;            // floats per chain row of leaf values: two chunk slots (one when resident)
    uint32_t off_lists, off_rec, off_frow, off_any, off_desc;
    uint32_t frow_stride;     // single-pass modes: bytes between the two feature-row buffers
};

// Leaf indices of four trees for this lane: nb holds the LDS byte addresses
// of the trees' node blocks (per lane), fb the lane's tile column.  The
// levels are those of the tree kernel's walk (five vector instructions per
// level and tree); trees are independent, so their LDS round trips overlap.
// The reads are issued with absolute LDS addresses from inline asm (the
// compiler would add the dynamic LDS base to every address) and waited for
// in the same statement.
template <int DEPTH>
__device__ __forceinline__ void walk4_local(const uint32_t (&nb)[4], uint32_t fb, uint32_t (&q)[4]) {
    uint32_t node[4], p[4], fa[4], pa[4];
    asm volatile(
        "ds_read_u16 %0, %4\n\t"
        "ds_read_u16 %1, %5\n\t"
        "ds_read_u16 %2, %6\n\t"
        "ds_read_u16 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(node[0]), "=&v"(node[1]), "=&v"(node[2]), "=&v"(node[3])
        : "v"(nb[0]), "v"(nb[1]), "v"(nb[2]), "v"(nb[3]));
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        p[g] = 1u;
        fa[g] = (node[g] & LOCAL_TILE_MASK) | fb;
        pa[g] = nb[g] + 4u;
    }
#pragma unroll
    for (int l = 0; l + 1 < DEPTH; ++l) {
        uint32_t x4[4], pr[4];
        asm volatile(
            "ds_read_u8 %0, %8\n\t"
            "ds_read_b32 %4, %12\n\t"
            "ds_read_u8 %1, %9\n\t"
            "ds_read_b32 %5, %13\n\t"
            "ds_read_u8 %2, %10\n\t"
            "ds_read_b32 %6, %14\n\t"
            "ds_read_u8 %3, %11\n\t"
            "ds_read_b32 %7, %15\n\t"
            "s_waitcnt lgkmcnt(0)"
            : "=&v"(x4[0]), "=&v"(x4[1]), "=&v"(x4[2]), "=&v"(x4[3]), "=&v"(pr[0]), "=&v"(pr[1]), "=&v"(pr[2]),
              "=&v"(pr[3])
            : "v"(fa[0]), "v"(fa[1]), "v"(fa[2]), "v"(fa[3]), "v"(pa[0]), "v"(pa[1]), "v"(pa[2]), "v"(pa[3]));
        const uint32_t mask = LOCAL_TILE_MASK;
        asm(AT_WALK4_ASM
            : "+v"(node[0]), "+v"(node[1]), "+v"(node[2]), "+v"(node[3]), "+v"(p[0]), "+v"(p[1]), "+v"(p[2]),
              "+v"(p[3]), "=&v"(fa[0]), "=&v"(fa[1]), "=&v"(fa[2]), "=&v"(fa[3]), "=&v"(pa[0]), "=&v"(pa[1]),
              "=&v"(pa[2]), "=&v"(pa[3])
            : "v"(x4[0]), "v"(x4[1]), "v"(x4[2]), "v"(x4[3]), "v"(pr[0]), "v"(pr[1]), "v"(pr[2]), "v"(pr[3]),
              "s"(mask), "v"(fb), "v"(nb[0]), "v"(nb[1]), "v"(nb[2]), "v"(nb[3])
            : "vcc");
    }
    uint32_t x4[4];
    asm volatile(
        "ds_read_u8 %0, %4\n\t"
        "ds_read_u8 %1, %5\n\t"
        "ds_read_u8 %2, %6\n\t"
        "ds_read_u8 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(x4[0]), "=&v"(x4[1]), "=&v"(x4[2]), "=&v"(x4[3])
        : "v"(fa[0]), "v"(fa[1]), "v"(fa[2]), "v"(fa[3]));
#pragma unroll
    for (int g = 0; g < 4; ++g) q[g] = 2u * p[g] + (x4[g] >= (node[g] & 0xffu) ? 1u : 0u) - (1u << DEPTH);
}

// Issues the direct-to-LDS loads of trees [t0, t0 + nt) of the local form
// into LDS at dst: thread li of nl (whole waves) moves 16-byte units
// li, li + nl, ...
__device__ __forceinline__ void load_trees(const LocalArgs& a, uint8_t* dst, int t0, int nt, int li, int nl) {
    const int n16 = (nt * a.ts * 4 + 15) >> 4;
    const uint4* src = reinterpret_cast<const uint4*>(a.tw + (size_t)t0 * a.ts);
    uint4* d = reinterpret_cast<uint4*>(dst);
    for (int base = li - (li & 63); base < n16; base += nl) {
        const int i = base + (li & 63);
        if (i < n16) __builtin_amdgcn_global_load_lds(src + i, d + base, 16, 0, 0);
    }
}


// Adds the leaf values row[0 .. nt) to s in order (row 16-byte aligned):
// blocks of sixteen float4 reads in flight, then their 64 adds; the rest in
// batches of 8, 4, 2 and 1 float4.  Nothing is carried from one block to
// the next but s, so the compiler has no registers to shuffle between
// blocks, and every branch is uniform (no selects in the chain of adds).
__device__ __forceinline__ void add4(float& s, const float4& v) {
    s = s + v.x;
    s = s + v.y;
    s = s + v.z;
    s = s + v.w;
}

template <int B>
__device__ __forceinline__ void fold_block(float& s, const float4* __restrict__ r4) {
    float4 R[B];
#pragma unroll
    for (int g = 0; g < B; ++g) R[g] = r4[g];
#pragma unroll
    for (int g = 0; g < B; ++g) add4(s, R[g]);
}

__device__ __forceinline__ float fold_row(float s, const float* __restrict__ row, int nt) {
    const float4* r4 = reinterpret_cast<const float4*>(row);
    const int n4 = nt >> 2;
    int i = 0;
    for (; i + 16 <= n4; i += 16) fold_block<16>(s, r4 + i);
    if (n4 - i >= 8) {
        fold_block<8>(s, r4 + i);
        i += 8;
    }
    if (n4 - i >= 4) {
        fold_block<4>(s, r4 + i);
        i += 4;
    }
    if (n4 - i >= 2) {
        fold_block<2>(s, r4 + i);
        i += 2;
    }
    if (n4 - i >= 1) fold_block<1>(s, r4 + i);
    for (int t = n4 * 4; t < nt; ++t) s = s + row[t];
    return s;
}

// The knob a step changes and the value it draws among the knob's other
// values, before the shift past the current value (block (chain, step, 0, 0)).
// Neither depends on the chain's state, so they are drawn ahead of time.
__device__ __forceinline__ void draw_move(const SpaceDesc& sd, uint32_t k0, uint32_t k1, uint32_t chain,
                                          uint32_t step, int& jm, uint32_t& v, uint64_t& radix) {
    const U4 rr = philox(k0, k1, U4{chain, step, 0u, 0u});
    jm = -1;
    v = 0u;
    radix = 0;
    if (sd.n_mut > 0) {
        jm = sd.mut[uniform_below(rr.x, (uint32_t)sd.n_mut)];
        v = uniform_below(rr.y, sd.knob_size[jm] - 1u);
        radix = sd.radix[jm];
    }
}

// base with knob jm moved to the drawn value v shifted past base's value
// (jm < 0: no knob can move), and the configuration index of the result.
__device__ __forceinline__ void apply_move(const uint32_t (&base)[MAX_KNOBS], uint64_t base_cfg, int jm, uint32_t v,
                                           uint64_t radix, uint32_t (&out)[MAX_KNOBS], uint64_t& cfg) {
    uint32_t old = 0;
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) {
        old = (j == jm) ? base[j] : old;
        out[j] = (j == jm) ? v + (v >= base[j] ? 1u : 0u) : base[j];
    }
    // the index moves by (new - old) times the knob's weight
    const uint32_t nv = v + (v >= old ? 1u : 0u);
    cfg = jm < 0 ? base_cfg
                 : (nv >= old ? base_cfg + (uint64_t)(nv - old) * radix : base_cfg - (uint64_t)(old - nv) * radix);
}

// FAST instances run the single-pass plans with at most four chains per
// workgroup and full workgroups (the launcher picks them); the others run
// every other plan.  Compiling the two apart keeps each one's uniform state
// within the scalar registers.
template <int TMPL, int DEPTH, bool FAST>
__global__ __launch_bounds__(LOCAL_WG_MAX) void k_local(LocalArgs a) {
    using N = Nest<TMPL>;
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
    uint32_t* s_any = reinterpret_cast<uint32_t*>(lds + a.off_any);   // [2]: some chain qualifies
    SpaceDesc& s_desc = *reinterpret_cast<SpaceDesc*>(lds + a.off_desc);
    uint64_t* s_fac = reinterpret_cast<uint64_t*>(lds + a.off_desc + sizeof(SpaceDesc));

    // LDS address of the dynamic block (0: the kernel has no static LDS, as
    // the launcher checks); the walk's and-or of node bits and the lane's
    // tile column needs the tile at a 16 KB boundary
    const uint32_t lbase = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)lds;
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
    // wave roles: 0 folds and keeps the books; 1 .. nww walk; the rest load
    const int nww = a.walk_waves;
    const bool walker = wave >= 1 && wave <= nww;
    const bool loader = wave > nww;
    const int n_load_waves = nthreads / 64 - 1 - nww;

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
    // space of the owner's chain: the staged copy in LDS or the set's tables
    // in global memory.  Each use branches on
    // `staged` (uniform in the workgroup) so that either branch reads one
    // address space directly.
    const SpaceDesc* sdp_g = a.descs + space_of(a.offsets, a.n_spaces, c);
    auto with_space = [&](auto&& f) {
        if (staged) f(s_desc);
        else f(*sdp_g);
    };

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
    if (tid < 2) s_any[tid] = 0u;
    const int rounds = (a.init ? 1 : 0) + a.steps;
    const bool resident = a.resident != 0 || a.tail != 0;
    const int nck = a.n_chunks;
    const int total_chunks = rounds * nck;
    const int lag = a.gather ? 2 : 1;   // chunks between a walk and the fold of its leaf values
    // the first chunk (every tree when resident) is loaded by all waves but 0
    if (wave >= 1 && rounds > 0) {
        load_trees(a, ring, 0, resident ? a.T : (a.ct < a.T ? a.ct : a.T), tid - 64, nthreads - 64);
        __builtin_amdgcn_s_waitcnt(0);
    }
    // the staged tables, initial lists and records are in place
    lds_barrier();

    // walker geometry: chain jw, tree slot u; a chunk of nt trees gives slot
    // u the trees u, u + S', u + 2S', u + 3S' with S' = ceil(nt / 4)
    const int wi = tid - 64;
    const int jw = lane % cpb;
    const int u = (walker ? wi : 0) / cpb;
    const uint32_t fb = lbase | (uint32_t)lane * 4u;
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    const uint32_t gchain = (uint32_t)(a.chain0 + (uint64_t)c);
    // the owner's next threshold and move, ready one round ahead (in tail
    // mode the threshold of each round after the first is brought into the
    // chain's record by the last wave during the previous fold)
    float thr_next = (owner && a.steps > 0) ? a.thr[c * a.steps] : 0.0f;
    int mv_j = -1;
    uint32_t mv_v = 0u;
    uint64_t mv_radix = 0;     // weight of the moved knob in the configuration index
    uint64_t cur_cfg = 0;      // index of the current configuration
    if (owner && !a.init)
        with_space([&](const SpaceDesc& sd) {
#pragma unroll
            for (int j = 0; j < MAX_KNOBS; ++j)
                if (j < sd.n_knobs) cur_cfg += (uint64_t)cur[j] * sd.radix[j];
        });
    if (owner && a.steps > 0)
        with_space([&](const SpaceDesc& sd) { draw_move(sd, k0, k1, gchain, a.step0, mv_j, mv_v, mv_radix); });
    // Fast plans (single pass, at most four chains per workgroup) take the
    // owners' side work off the path from one fold to the next: a helper
    // wave draws the moves two steps ahead, and a round's candidates are
    // offered to the best lists by another wave during the next round's fold
    // (the offers of a chain stay in round order).  Roles during a fold:
    // wave 0 folds, waves 1-2 make and evaluate the next candidates, wave 3
    // offers, wave 4 draws, the last wave brings the next thresholds.  The
    // chain's record carries, by round parity, the two candidates made for
    // the round, which of them is the round's (the previous accept's
    // outcome) and the configuration the round starts from, so that no
    // reader in one round meets a writer of the same round.
    // single pass: every tree walked in one pass per round (tail mode, or
    // resident trees in one chunk); such runs work a round ahead
    const bool single = FAST || a.tail || (a.resident && a.n_chunks == 1);
    const bool fast = FAST;
    auto draw_into = [&](int j, int st) {
        // move of step st for chain j into its record (slot st & 1)
        int jm;
        uint32_t v;
        uint64_t radix;
        const uint32_t gch = (uint32_t)(a.chain0 + (uint64_t)(c0 + j));
        if (staged) draw_move(s_desc, k0, k1, gch, a.step0 + (uint32_t)st, jm, v, radix);
        else draw_move(a.descs[space_of(a.offsets, a.n_spaces, c0 + j)], k0, k1, gch, a.step0 + (uint32_t)st, jm, v,
                       radix);
        rec[j].mvj[st & 1] = jm;
        rec[j].mvv[st & 1] = v;
        rec[j].mvr[st & 1] = radix;
    };
    // offer of round rr's candidates (waiting in the records) by the 16-lane
    // groups of one wave: group g takes chain g
    auto offer_pending = [&](int rr) {
        const int g = lane >> 4, gl = lane & 15;
        const int jc = g < nc ? g : 0;
        ChainRec& R = rec[jc];
        const uint64_t pc = R.pcfg[rr & 1];
        const float ps = R.pscore[rr & 1];
        const bool first = a.init && rr == 0;
        const bool q = g < nc && (first || (int)R.count < k || precedes(ps, pc, R.kth_score, R.kth_cfg));
        if (gl == 0 && g < nc) {
            R.cfg = pc;
            R.score = ps;
        }
        group_offer(lists + jc * k, R, k, gl, 0xffffull << (16 * g), q);
    };
    if (fast && owner) {
        const int s1 = (a.init ? -1 : 0) + 1;
        if (s1 < a.steps) draw_into(tid, s1);
        // round 0 starts from the loaded configuration; its candidate is
        // outcome 0
        ChainRec& R = rec[tid];
#pragma unroll
        for (int j = 0; j < MAX_KNOBS / 2; ++j) R.curk[0][j] = cur[2 * j] | (cur[2 * j + 1] << 16);
        R.curcfg[0] = cur_cfg;
        R.ssel[0] = 0u;
    }

    // Loop gr's features of chain j's configuration nx into row dst.
    auto eval_loop = [&](const uint32_t (&nx)[MAX_KNOBS], int j, int gr_, uint8_t* dst) {
        auto feats = [&](const SpaceDesc& sd, const uint64_t* facp) {
            uint32_t fac[6][4];
            gather_factors<TMPL>(sd, facp, nx, fac);
            uint32_t f[11];
            loop_features<TMPL>(sd, fac, ann_knobs_of<TMPL>(sd, nx), gr_, f);
#pragma unroll
            for (int i = 0; i < 11; ++i) dst[gr_ * 11 + i] = (uint8_t)f[i];
        };
        if (staged) feats(s_desc, s_fac);
        else feats(a.descs[space_of(a.offsets, a.n_spaces, c0 + j)], a.factors);
    };
    auto unpack = [](const uint32_t (&w)[MAX_KNOBS / 2], uint32_t (&nx)[MAX_KNOBS]) {
#pragma unroll
        for (int j = 0; j < MAX_KNOBS; ++j) nx[j] = (w[j >> 1] >> (16 * (j & 1))) & 0xffffu;
    };
    // single-pass plans work a round ahead: while a round's scores are
    // folded, the other waves evaluate the next round's candidate both for
    // an accepted and for a rejected current one (feature rows 0 and 1), so
    // a round starts from ready rows.
    const int cpb_log2 = __builtin_ctz((unsigned)cpb);
    uint32_t cd[MAX_KNOBS];
    uint64_t cfg = 0;
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) cd[j] = 0u;
    for (int r = 0; r < rounds; ++r) {
        const bool is_init = a.init && r == 0;
        const int s = r - (a.init ? 1 : 0);
        const bool ahead = single && r > 0;   // this round's candidate and rows are ready
        const bool more = r + 1 < rounds;
        // (1) candidate: the initial draw (block (chain, 0, 1, j / 4)) or one
        // knob moved to a uniformly chosen other value
        float thr_v = 0.0f;
        if (owner && ahead) {
            thr_v = rec[tid].thr;
            if (fast) {
                // the candidate evaluated for this round's outcome
                const ChainRec& R = rec[tid];
                const uint32_t os = R.ssel[r & 1] & 1u;
                uint32_t w[MAX_KNOBS / 2];
#pragma unroll
                for (int j = 0; j < MAX_KNOBS / 2; ++j) w[j] = R.snx[r & 1][os][j];
                unpack(w, cd);
                cfg = R.scfg[r & 1][os];
            }
        } else if (owner) {
            cfg = 0;
            if (is_init) {
                with_space([&](const SpaceDesc& sd) {
                    U4 rr{0, 0, 0, 0};
#pragma unroll
                    for (int j = 0; j < MAX_KNOBS; ++j) {
                        if ((j & 3) == 0) rr = philox(k0, k1, U4{gchain, 0u, 1u, (uint32_t)(j >> 2)});
                        const uint32_t word = (j & 3) == 0 ? rr.x : (j & 3) == 1 ? rr.y : (j & 3) == 2 ? rr.z : rr.w;
                        cd[j] = (j < sd.n_knobs) ? uniform_below(word, sd.knob_size[j]) : 0u;
                        if (j < sd.n_knobs) cfg += (uint64_t)cd[j] * sd.radix[j];
                    }
                });
            } else {
                thr_v = thr_next;
                if (s + 1 < a.steps) thr_next = a.thr[c * a.steps + s + 1];
                apply_move(cur, cur_cfg, mv_j, mv_v, mv_radix, cd, cfg);
            }
#pragma unroll
            for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].nx[j] = cd[2 * j] | (cd[2 * j + 1] << 16);
            if (fast) {
#pragma unroll
                for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].snx[r & 1][0][j] = rec[tid].nx[j];
                rec[tid].scfg[r & 1][0] = cfg;
            }
        }
        if (!ahead) {
            lds_barrier();
            // (2) features: lane gr of group gj evaluates loop gr of chain gj
            if (gvalid && gr < N::L) {
                uint32_t nx[MAX_KNOBS];
                unpack(rec[gj].nx, nx);
                eval_loop(nx, gj, gr, frow + gj * RS);
            }
            lds_barrier();
        }
        // (3) the tile: column l holds chain l % cpb (the last chain stands
        // in for missing ones), bytes 4x+3
        // (features are at most 31, so 4x+3 stays within each byte; bytes past
        // the last feature are never read)
        if (!single || wave > 0) {
            // In tail mode waves 1.. fill the tile while the owners in wave 0
            // prepare the next candidates; else every wave does.  Thread t of
            // the fill fills tile words t, t + NF, ...: always chain t % cpb
            // (cpb divides NF, 448 or 512).
            constexpr int NF_MIN = LOCAL_WG_MAX - 64;
            constexpr int TU = (Q * 64 + NF_MIN - 1) / NF_MIN;
            const int nf = single ? nthreads - 64 : nthreads;
            const int t = single ? tid - 64 : tid;
            int j = t & (cpb - 1);
            j = j < nc ? j : nc - 1;
            uint32_t w[TU];
            if (fast) {
                // 448 fill threads: the words of every pass but the last exist
                const uint8_t* row = frow + (ahead ? (rec[j].ssel[r & 1] & 1u) * a.frow_stride : 0u) + j * RS;
                constexpr bool LAST = (TU - 1) * NF_MIN + NF_MIN > Q * 64;   // the last pass is partial
                const bool last_ok = !LAST || t + (TU - 1) * NF_MIN < Q * 64;
#pragma unroll
                for (int u = 0; u < TU; ++u)
                    if (u + 1 < TU || last_ok)
                        w[u] = *reinterpret_cast<const uint32_t*>(row + 4 * ((t + u * NF_MIN) >> 6));
#pragma unroll
                for (int u = 0; u < TU; ++u)
                    if (u + 1 < TU || last_ok) tile[t + u * NF_MIN] = (w[u] << 2) | 0x03030303u;
            } else {
                const uint8_t* row = frow + (ahead ? rec[j].sel * a.frow_stride : 0u) + j * RS;
#pragma unroll
                for (int u = 0; u < TU; ++u) {
                    const int i = t + u * nf;
                    if (i < Q * 64) w[u] = *reinterpret_cast<const uint32_t*>(row + 4 * (i >> 6));
                }
#pragma unroll
                for (int u = 0; u < TU; ++u) {
                    const int i = t + u * nf;
                    if (i < Q * 64) tile[i] = (w[u] << 2) | 0x03030303u;
                }
            }
        }
        float sc = 0.0f;
        if (single) {
            // (4') every tree of every chain in one pass: in tail mode the
            // resident top levels from LDS, then the last level and its leaf
            // from the tree's 16-byte tail record; else the whole tree from
            // LDS.  Thread t takes chain t % cpb and, with S = min(ceil(T /
            // 4), threads / cpb) slots, slot u = t / cpb < S takes trees u,
            // u + S, u + 2S, u + 3S per pass.
            if (owner && more && !fast) {
                with_space([&](const SpaceDesc& sd) {
                    draw_move(sd, k0, k1, gchain, a.step0 + (uint32_t)(s + 1), mv_j, mv_v, mv_radix);
                });
                // the next candidate after an accept (from cd) and after a
                // reject (from cur; after the initial draw, which is always
                // accepted, also from cd), kept in the chain's record
                uint32_t nx[MAX_KNOBS];
                uint64_t ncfg;
                apply_move(cd, cfg, mv_j, mv_v, mv_radix, nx, ncfg);
#pragma unroll
                for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].nx[j] = nx[2 * j] | (nx[2 * j + 1] << 16);
                rec[tid].cfga = ncfg;
                if (is_init) apply_move(cd, cfg, mv_j, mv_v, mv_radix, nx, ncfg);
                else apply_move(cur, cur_cfg, mv_j, mv_v, mv_radix, nx, ncfg);
#pragma unroll
                for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].nxb[j] = nx[2 * j] | (nx[2 * j + 1] << 16);
                rec[tid].cfgb = ncfg;
            }
            lds_barrier();
            // (tail mode keeps every slot busy: its last-level gathers, not
            // the walks, set the pace)
            const int want = (a.T + 3) >> 2, have = nthreads / cpb;
            const int S = (a.tail || want > have) ? have : want;
            const int ua = tid / cpb;
            const int ja = tid & (cpb - 1);
            const uint32_t fba = lbase | (uint32_t)lane * 4u;
            auto trees_of = [&](int base, int (&ti)[4], uint32_t (&nb)[4]) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int t = base + ua + g * S;
                    ti[g] = t < a.T ? t : -1;
                    nb[g] = lbase + a.off_ring + (uint32_t)(t < a.T ? t : 0) * (uint32_t)a.ts * 4u;
                }
            };
            if (a.tail) {
                for (int base = 0; base < a.T; base += 4 * S) {
                    uint32_t nb[4], q[4];
                    int ti[4];
                    trees_of(base, ti, nb);
                    walk4_local<(DEPTH >= 2 ? DEPTH - 1 : 1)>(nb, fba, q);
                    uint4 rec4[4];
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int t = ti[g] >= 0 ? ti[g] : 0;
                        rec4[g] = a.tail_rec[((size_t)t << (DEPTH - 1)) + q[g]];
                    }
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const uint32_t node = rec4[g].x;
                        const uint32_t x4 = lds[((node & LOCAL_TILE_MASK) | fba) - lbase];
                        const uint32_t v = x4 >= (node & 0xffu) ? rec4[g].z : rec4[g].y;
                        if (ti[g] >= 0 && ja < nc) lv[ja * a.lv_stride + ti[g]] = __uint_as_float(v);
                    }
                }
            } else if (ua < S) {
                for (int base = 0; base < a.T; base += 4 * S) {
                    uint32_t nb[4], q[4];
                    int ti[4];
                    trees_of(base, ti, nb);
                    walk4_local<DEPTH>(nb, fba, q);
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const uint32_t v = *reinterpret_cast<const uint32_t*>(lds + (nb[g] - lbase) + NBB + 4u * q[g]);
                        if (ti[g] >= 0 && ja < nc) lv[ja * a.lv_stride + ti[g]] = __uint_as_float(v);
                    }
                }
            }
            lds_barrier();
            if (wave == 0) {
                if (lane < nc) sc = fold_row(sc, lv + lane * a.lv_stride, a.T);
            } else {
                if (fast && wave == 3 && r > 0) offer_pending(r - 1);
                if (fast && wave == 4 && lane < nc && s + 2 < a.steps) draw_into(lane, s + 2);
            }
            if (wave > 0 && more) {
                if (wave == nthreads / 64 - 1 && lane < nc) rec[lane].thr = a.thr[(c0 + lane) * a.steps + s + 1];
                // the next round's feature rows: item (v * cpb + j) * 16 + gr
                // is loop gr of chain j's candidate for outcome v
                for (int it = tid - 64; it < 32 * cpb; it += nthreads - 64) {
                    const int gr2 = it & 15, j = (it >> 4) & (cpb - 1), v = (it >> 4) >> cpb_log2;
                    if (j < nc && gr2 < N::L) {
                        uint32_t nx[MAX_KNOBS];
                        if (fast) {
                            // the candidate itself: step s + 1's move applied to
                            // this round's candidate (v = 0; also v = 1 after
                            // the initial draw, which is always accepted) or to
                            // the configuration the round started from (v = 1)
                            ChainRec& R = rec[j];
                            const int sl = (s + 1) & 1;
                            const uint32_t os = R.ssel[r & 1] & 1u;
                            uint32_t w[MAX_KNOBS / 2], base[MAX_KNOBS];
                            uint64_t bcfg;
                            if (v == 0 || is_init) {
#pragma unroll
                                for (int q = 0; q < MAX_KNOBS / 2; ++q) w[q] = R.snx[r & 1][os][q];
                                bcfg = R.scfg[r & 1][os];
                            } else {
#pragma unroll
                                for (int q = 0; q < MAX_KNOBS / 2; ++q) w[q] = R.curk[r & 1][q];
                                bcfg = R.curcfg[r & 1];
                            }
                            unpack(w, base);
                            uint64_t ncfg;
                            apply_move(base, bcfg, R.mvj[sl], R.mvv[sl], R.mvr[sl], nx, ncfg);
                            if (gr2 == 0) {
#pragma unroll
                                for (int q = 0; q < MAX_KNOBS / 2; ++q)
                                    R.snx[(r + 1) & 1][v][q] = nx[2 * q] | (nx[2 * q + 1] << 16);
                                R.scfg[(r + 1) & 1][v] = ncfg;
                            }
                        } else {
                            unpack(v ? rec[j].nxb : rec[j].nx, nx);
                        }
                        eval_loop(nx, j, gr2, frow + v * a.frow_stride + j * RS);
                    }
                }
            }
        } else {
        // (4) chunk pipeline.  Iteration it: loaders bring chunk it + 1;
        // walkers walk chunk it and write its leaf values (leaves gathered
        // from global memory are written one iteration later); wave 0 folds
        // chunk it - lag.
        uint32_t vprev[4] = {0u, 0u, 0u, 0u};
        int tprev[4] = {-1, -1, -1, -1};
        for (int it = 0; it < nck + lag; ++it) {
            const int gc = r * nck + it;
            if (loader && it < nck) __builtin_amdgcn_s_waitcnt(0);   // chunk it has landed
            lds_barrier();
            if (loader) {
                if (!resident && it < nck && gc + 1 < total_chunks) {
                    const int x = (it + 1) % nck;
                    const int t0 = x * a.ct;
                    load_trees(a, ring + (size_t)((gc + 1) & 1) * a.ring_bytes, t0,
                               (a.T - t0 < a.ct ? a.T - t0 : a.ct), tid - 64 * (1 + nww), 64 * n_load_waves);
                }
            } else if (walker) {
                const int t0 = it * a.ct;
                const int nt = it < nck ? (a.T - t0 < a.ct ? a.T - t0 : a.ct) : 0;
                const int sp4 = (nt + 3) >> 2;
                int ti[4] = {-1, -1, -1, -1};
                uint32_t nb[4], q[4];
                const bool walks = u < sp4;
                if (walks) {
                    // resident trees sit at their own place, streamed ones in buffer gc & 1
                    const uint32_t rb = lbase + a.off_ring + (resident ? (uint32_t)t0 * (uint32_t)a.ts * 4u
                                                                       : (uint32_t)(gc & 1) * a.ring_bytes);
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int tl = u + g * sp4;
                        ti[g] = tl < nt ? tl : -1;
                        nb[g] = rb + (uint32_t)(tl < nt ? tl : u) * (uint32_t)a.ts * 4u;
                    }
                    walk4_local<DEPTH>(nb, fb, q);
                }
                if (a.gather) {
                    // the leaf values gathered last iteration, then this chunk's
                    if (it > 0 && jw < nc) {
                        float* lvk = lv + ((it - 1) & 1) * a.ct + jw * a.lv_stride;
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            if (tprev[g] >= 0) lvk[tprev[g]] = __uint_as_float(vprev[g]);
                    }
                    if (walks) {
#pragma unroll
                        for (int g = 0; g < 4; ++g) {
                            const int tt = ti[g] >= 0 ? ti[g] : u;
                            vprev[g] = a.leaf_src[(size_t)(t0 + tt) * a.w16 + (NBB / 4) + q[g]];
                        }
                    }
#pragma unroll
                    for (int g = 0; g < 4; ++g) tprev[g] = walks ? ti[g] : -1;
                } else if (walks && jw < nc) {
                    float* lvk = lv + (it & 1) * a.ct + jw * a.lv_stride;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const uint32_t v = *reinterpret_cast<const uint32_t*>(lds + (nb[g] - lbase) + NBB + 4u * q[g]);
                        if (ti[g] >= 0) lvk[ti[g]] = __uint_as_float(v);
                    }
                }
            } else {
                if (it == 0 && owner && s + 1 < a.steps)
                    with_space([&](const SpaceDesc& sd) {
                        draw_move(sd, k0, k1, gchain, a.step0 + (uint32_t)(s + 1), mv_j, mv_v, mv_radix);
                    });
                const int fc = it - lag;   // chunk to fold
                if (fc >= 0 && lane < nc) {
                    const int t0 = fc * a.ct;
                    const int nt = a.T - t0 < a.ct ? a.T - t0 : a.ct;
                    sc = fold_row(sc, lv + lane * a.lv_stride + (fc & 1) * a.ct, nt);
                }
            }
        }
        }
        // (5) offer to the best list when some chain qualifies, then the
        // Metropolis test
        if (fast) {
            // only the outcome is needed before the barrier (the next round's
            // tile copy reads it); in tail mode the rest of the owner's books
            // follow it, beside the other waves' copy (in the resident mode
            // wave 0 walks first, so they stay ahead of it)
            const bool acc = owner && (is_init || (sc - cur_s) >= thr_v);
            if (owner) rec[tid].ssel[(r + 1) & 1] = acc ? 0u : 1u;
            auto books = [&]() {
                if (!is_init && a.trace) {
                    at_entry tr;
                    tr.cfg = cfg;
                    tr.score = sc;
                    tr.flag = acc ? 1u : 0u;
                    a.trace[c * a.steps + s] = tr;
                }
                // the candidate waits for its offer (wave 3, next round); the
                // next round starts from the configuration published here
                ChainRec& R = rec[tid];
                R.pcfg[r & 1] = cfg;
                R.pscore[r & 1] = sc;
                if (acc) {
#pragma unroll
                    for (int j = 0; j < MAX_KNOBS; ++j) cur[j] = cd[j];
                    cur_s = sc;
                    cur_cfg = cfg;
                }
#pragma unroll
                for (int j = 0; j < MAX_KNOBS / 2; ++j) R.curk[(r + 1) & 1][j] = cur[2 * j] | (cur[2 * j + 1] << 16);
                R.curcfg[(r + 1) & 1] = cur_cfg;
            };
            if (owner && !a.tail) books();
            lds_barrier();
            if (owner && a.tail) books();
            continue;
        }
        if (owner) {
            ChainRec& R = rec[tid];
            const bool qual = is_init || (int)R.count < k || precedes(sc, cfg, R.kth_score, R.kth_cfg);
            R.cfg = cfg;
            R.score = sc;
            R.qual = qual ? 1u : 0u;
            // the next round's rows (read after the barrier below)
            R.sel = (is_init || (sc - cur_s) >= thr_v) ? 0u : 1u;
            if (qual) atomicOr(&s_any[r & 1], 1u);
        }
        if (tid == 0) s_any[(r + 1) & 1] = 0u;
        lds_barrier();
        if (s_any[r & 1]) {
            if (gj < cpb) group_offer(lists + gjc * k, rec[gjc], k, gr, gmask, gvalid && rec[gjc].qual != 0);
            lds_barrier();
        }
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
                cur_cfg = cfg;
            }
            if (single && more) {
                const ChainRec& R = rec[tid];
                unpack(acc ? R.nx : R.nxb, cd);
                cfg = acc ? R.cfga : R.cfgb;
            }
        }
    }

    // the last round's offer, once the owners have recorded its candidates
    if (fast && rounds > 0) {
        lds_barrier();
        if (wave == 3) offer_pending(rounds - 1);
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

template <int TMPL, bool FAST>
hipError_t launch_local_t(const LocalArgs& a, int depth, int grid, int threads, size_t lds, hipStream_t stream,
                          hipEvent_t start, hipEvent_t stop) {
    const void* fn = nullptr;
    switch (depth) {
#define AT_LOCAL_CASE(D) \
    case D: fn = reinterpret_cast<const void*>(&k_local<TMPL, D, FAST>); break;
        AT_LOCAL_CASE(1) AT_LOCAL_CASE(2) AT_LOCAL_CASE(3) AT_LOCAL_CASE(4) AT_LOCAL_CASE(5) AT_LOCAL_CASE(6)
        AT_LOCAL_CASE(7) AT_LOCAL_CASE(8) AT_LOCAL_CASE(9) AT_LOCAL_CASE(10) AT_LOCAL_CASE(11) AT_LOCAL_CASE(12)
#undef AT_LOCAL_CASE
        default: return hipErrorInvalidValue;
    }
    static bool configured[13] = {};
    if (!configured[depth]) {
        // the walk addresses the tile with an and-or, which needs the
        // dynamic LDS block at address 0: no static LDS in the kernel
        hipFuncAttributes fa;
        hipError_t e = hipFuncGetAttributes(&fa, fn);
        if (e != hipSuccess) return e;
        if (fa.sharedSizeBytes != 0) return hipErrorInvalidKernelFile;
        e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)LOCAL_LDS_BYTES);
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
// Workgroups of 512 threads: wave 0 folds and keeps the books, then walker
// waves (a slot per chain and up to four trees per slot and chunk), then
// loader waves.  Chains per workgroup: the smallest divisor of 64 that
// leaves at most one workgroup per compute unit (at most 32).  A streamed
// chunk leaves at least four loader waves when it can: one wave moves about
// 8 bytes per clock from L2, a compute unit some 50-60.
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
    const int threads = 512, waves = threads / 64;
    // trees per chunk that w walker waves cover (four per slot), a multiple of 4
    auto walk_cap = [&](int w) { return 4 * (w * 64 / cpb) / 4 * 4; };
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
                         al16((size_t)cpb * RS) + 16 + al16(sizeof(SpaceDesc) + (size_t)fac_max * 8);
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
    const int cap_all = walk_cap(waves - 1);
    const int ct_res = T <= cap_all ? T : cap_all;
    const size_t res_bytes = al16((size_t)T * ts_full * 4);
    // tail: the tree tops (levels 0 .. d-2) resident, every tree walked in
    // one pass with the last level and leaf read from the tail records;
    // needs one row of leaf values per chain for all trees
    const int ts_top = local_tree_stride(d >= 2 ? NB / 2 : 1);
    const size_t top_bytes = al16((size_t)T * ts_top * 4);
    const int T4 = (T + 3) / 4 * 4;
    const size_t lv_all = al16((size_t)cpb * ((size_t)T4 + 4) * 4);
    // (one chunk of resident trees also needs a second feature-row buffer)
    if (cap_all >= 4 && res_bytes + lv_bytes(ct_res) + (ct_res == T ? al16((size_t)cpb * RS) : 0) <= avail) {
        pl.resident = 1;
        pl.gather = 0;
        pl.ts = ts_full;
        pl.ct = ct_res;
        pl.ring_bytes = (uint32_t)res_bytes;
    } else if (d >= 2 && top_bytes + lv_all + al16((size_t)cpb * RS) <= avail) {
        pl.tail = 1;
        pl.resident = 0;
        pl.gather = 0;
        pl.ts = ts_top;
        pl.ct = T;
        pl.ring_bytes = (uint32_t)top_bytes;
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
        const int cap = walk_cap(3) >= 16 ? walk_cap(3) : walk_cap(waves - 2);
        ct_max = ct_max < cap ? ct_max : cap;
        if (ct_max < 4) return false;
        const int chunks = (T + ct_max - 1) / ct_max;
        pl.ct = ((T + chunks - 1) / chunks + 3) / 4 * 4;
        pl.ring_bytes = (uint32_t)al16((size_t)pl.ct * pl.ts * 4);
    }
    pl.walk_waves = (pl.ct * cpb + 255) / 256;
    if (pl.walk_waves > waves - 1) pl.walk_waves = waves - 1;
    pl.n_chunks = (T + pl.ct - 1) / pl.ct;
    pl.lv_stride = pl.tail ? T4 + 4 : 2 * pl.ct + 4;
    size_t off = tile + ((pl.resident || pl.tail) ? 1 : 2) * (size_t)pl.ring_bytes;
    pl.off_lv = (uint32_t)off;
    off += pl.tail ? lv_all : lv_bytes(pl.ct);
    pl.off_lists = (uint32_t)off;
    off += al16((size_t)cpb * ch.topk * sizeof(at_entry));
    pl.off_rec = (uint32_t)off;
    off += al16((size_t)cpb * sizeof(ChainRec));
    pl.off_frow = (uint32_t)off;
    // single-pass modes (tail, one resident chunk): two buffers, the next
    // round's rows for an accepted and for a rejected candidate
    pl.frow_stride = (pl.tail || (pl.resident && pl.n_chunks == 1)) ? (uint32_t)al16((size_t)cpb * RS) : 0u;
    off += al16((size_t)cpb * RS) + pl.frow_stride;
    pl.off_any = (uint32_t)off;
    off += 16;
    pl.off_desc = (uint32_t)off;
    off += al16(sizeof(SpaceDesc) + (size_t)fac_max * 8);
    pl.lds_bytes = off;
    // streamed bytes per round and workgroup, for the path choice
    pl.round_bytes = pl.resident ? 0.0
                   : pl.tail ? (double)cpb * T * 64
                             : (double)T * pl.ts * 4 + (pl.gather ? (double)cpb * T * 64 : 0.0);
    return pl.lds_bytes <= LOCAL_LDS_BYTES;
}

hipError_t launch_sa_local(const at_space_s& sp, const EnsembleDesc& e, at_chains_s& ch, const LocalPlan& pl,
                           int steps, bool init, const float* thr, at_entry* best, at_entry* trace,
                           hipStream_t stream) {
    const int64_t n = ch.n_chains;
    if (n == 0) return hipSuccess;
    // the kernel's tile fill and its wave roles assume full workgroups
    if (pl.threads != LOCAL_WG_MAX) return hipErrorInvalidConfiguration;
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
    a.tw = pl.tail ? e.local_top : (pl.gather ? e.local_nodes : e.local_full);
    a.ts = pl.ts;
    a.T = e.n_trees;
    a.ct = pl.ct;
    a.n_chunks = pl.n_chunks;
    a.resident = pl.resident;
    a.tail = pl.tail;
    a.tail_rec = e.tail;
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
    a.frow_stride = pl.frow_stride;
    a.off_any = pl.off_any;
    a.walk_waves = pl.walk_waves;
    a.off_desc = pl.off_desc;
    ch.events_used[0] = ch.events_used[1] = 0;
    hipEvent_t start = nullptr, stop = nullptr;
    if ((err = next_events(ch, 0, start, stop)) != hipSuccess) return err;
    const bool fast = (pl.tail || (pl.resident && pl.n_chunks == 1)) && pl.cpb <= 4 && pl.threads == LOCAL_WG_MAX;
    if (sp.tmpl == AT_TMPL_GEMM)
        return fast ? launch_local_t<AT_TMPL_GEMM, true>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream, start,
                                                         stop)
                    : launch_local_t<AT_TMPL_GEMM, false>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream, start,
                                                          stop);
    return fast ? launch_local_t<AT_TMPL_CONV2D_NCHW, true>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream,
                                                            start, stop)
                : launch_local_t<AT_TMPL_CONV2D_NCHW, false>(a, e.depth, pl.grid, pl.threads, pl.lds_bytes, stream,
                                                             start, stop);
}

}  // namespace at
