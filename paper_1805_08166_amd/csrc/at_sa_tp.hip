// Parallel simulated annealing (Section 3.3), tree-partitioned across the GPU.
//
// One annealing step of every chain is two kernels:
//   k_chain  one lane per chain: folds the leaf values of the candidate just
//            scored (tree order, fp32, from +0.0f), offers it to the chain's
//            best list, applies the Metropolis test, then publishes the next
//            candidate (one knob changed, Philox block (chain, step, 0, 0))
//            and its loop-context features as packed bytes 4x+3,
//            quad-major (dword q of chain c at Fg[q * n + c]).  The next
//            candidates of both outcomes of the test, and their features,
//            are built by the workgroup's other waves while the fold runs.
//   k_trees  workgroup w holds the pointer form of trees [w*tpw, (w+1)*tpw)
//            in LDS; each of its waves walks them for 64 chains at a time
//            through its own LDS feature tile, writing the reached leaf
//            values to V.
// The kernel boundary is the only device-wide synchronisation: it is cheaper
// than an in-kernel grid barrier here because the cross-XCD data (features
// and leaf values) must be written back from the per-XCD L2 caches anyway.
//
// V is laid out by blocks of 16 chains, then groups of four trees: the
// values of trees 4g..4g+3 for chain c are the 16 bytes at float
// ((c / 16) * G + g) * 64 + (c % 16) * 4 with G = ceil(T / 4) groups, so a
// chain kernel workgroup (16 chains) reads one contiguous stretch of V and
// the fold reads one float4 per lane per group.
#include <cstddef>

#include <hip/hip_ext.h>

#include "at_chain.h"

namespace at {
namespace {

using namespace dev;

// Float index of tree t's leaf value for chain c in V (groups: ceil(T / 4)).
__device__ __forceinline__ int64_t v_index(int64_t c, int t, int groups) {
    return ((((c >> 4) * groups + (t >> 2)) << 6) + ((c & 15) << 2) + (t & 3));
}

// Chain-kernel workgroups have 256 or 512 threads (template argument
// CHAIN_WG): wave 0 folds, the others build the next candidates (see
// launch_sa_tp for the choice).
constexpr int CPW = 16;                 // chains per chain-kernel workgroup
static_assert(CPW == 16 && CPW == STAGE_CHAINS, "a chain-kernel workgroup reads one 16-chain block of V");
constexpr int FOLD_P = 32;              // 4-tree groups per fold pass: 32 x 16 chains x 16 B = 8 KB
// Passes in the LDS ring: one model's fold keeps one pass in flight while
// it adds the other (deeper rings measured slower: C12 chain kernel 16.3 us
// with two passes, 16.6 with three, 16.7 with four, 17.1 with six); Eq. 4's
// two folds take a pass of each at a time and keep a pair in flight.
constexpr int FOLD_R1 = 2;
constexpr int FOLD_R2 = 4;
constexpr size_t PASS_BYTES = (size_t)FOLD_P * CPW * 16;
__host__ __device__ constexpr size_t ring_bytes(bool two_models) {
    return (two_models ? FOLD_R2 : FOLD_R1) * PASS_BYTES;
}
constexpr int KMAX = 64;                // largest best list
constexpr size_t MAX_LDS_BYTES = 163840; // LDS of one compute unit

enum { FIN_NONE = 0, FIN_INIT = 1, FIN_STEP = 2 };
enum { DRAW_NONE = 0, DRAW_INIT = 1, DRAW_PROPOSE = 2 };

struct ChainArgs {
    const SpaceDesc* descs;
    const int64_t* offsets;
    int n_spaces;
    const uint64_t* factors;
    // LDS images of the spaces (descriptor rebased, then split factors),
    // stage_stride bytes apart; the image of a workgroup's chains is
    // stage_single (one space) or wg_space[workgroup] (sets), -1 for none
    const uint8_t* stage;
    int stage_stride;
    int stage_single;
    const int32_t* wg_space;
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
    uint32_t* Fg;             // [Q][fg_stride] packed features
    int64_t fg_stride;        // n rounded up to 64 chains
    int fin;                  // what the pending candidate is
    int fin_step;             // its local step index (thr / trace row)
    int steps;                // row length of thr and trace
    const float* thr;
    at_entry* trace;
    int draw;                 // what to propose next
    uint32_t draw_step;       // absolute step of the proposal
    at_entry* best;           // copy of the best lists (last launch), or null
    // Eq. 4 runs: leaf values of the global model (over the candidates'
    // relation features), folded before the local model's V and added to
    // its sum; the candidates' relation features go to Fr as packed bytes,
    // quad-major ([REL_Q][fg_stride]).  Null for one-model runs.
    const float* Vg;
    int Tg;
    uint32_t* Fr;
    // trees of the next tree launch, relocated (pf_tree_bytes each, pf_tpw
    // a tree workgroup, pf_trees in all): the building waves bring them
    // into their XCD's L2 before the tree kernel copies them; null: none
    const uint8_t* pf_trees;
    int pf_tree_bytes;
    int pf_tpw;
    int pf_ntrees;
    // tile layout of Fg: fq quads, position p holding loop-context feature
    // fsrc[p] (0xff: padding); fident: position p holds feature p
    const uint8_t* fsrc;
    int fq;
    int fident;
};

constexpr int REL_F = 192;              // context relation features per candidate
constexpr int REL_Q = REL_F / 4;


// Batches of FOLD_B groups (stride CPW float4 in the ring): the reads of a
// batch, then its adds in tree order.
constexpr int FOLD_B = 8;
__device__ __forceinline__ void fold_load(float4 (&R)[FOLD_B], const float4* __restrict__ src) {
#pragma unroll
    for (int g = 0; g < FOLD_B; ++g) R[g] = src[g * CPW];
}

__device__ __forceinline__ void fold_add(float& s, const float4 (&R)[FOLD_B]) {
#pragma unroll
    for (int g = 0; g < FOLD_B; ++g) {
        s = s + R[g].x;
        s = s + R[g].y;
        s = s + R[g].z;
        s = s + R[g].w;
    }
}

// A whole pass (FOLD_P groups) added in order, two register sets deep: the
// reads of batch b + 1 are in flight while batch b is added (a dependent
// fp32 add takes about as long as ten issue slots, an LDS read several
// adds).  The reads are issued from inline asm at the lane's LDS byte
// address and waited for explicitly: LDS reads of one wave complete in
// order, so at most FOLD_B outstanding means the older batch has landed
// (other outstanding LDS or scalar operations only make the wait longer).
// Each wait statement takes its batch's registers as operands, so no add
// can move ahead of it.
static_assert(FOLD_P == 4 * FOLD_B && FOLD_B == 8, "a pass is four batches of eight reads");
typedef float fold_v4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_byte_address(const void* p) {
    // the LDS aperture's base has zero low 32 bits
    return (uint32_t)reinterpret_cast<uintptr_t>(p);
}

template <int OFF>
__device__ __forceinline__ void fold_issue_batch(fold_v4 (&R)[FOLD_B], uint32_t ad) {
#define AT_FOLD_READ(G) \
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(R[G]) : "v"(ad), "i"(OFF + (G) * CPW * 16))
    AT_FOLD_READ(0);
    AT_FOLD_READ(1);
    AT_FOLD_READ(2);
    AT_FOLD_READ(3);
    AT_FOLD_READ(4);
    AT_FOLD_READ(5);
    AT_FOLD_READ(6);
    AT_FOLD_READ(7);
#undef AT_FOLD_READ
}

#define AT_FOLD_WAIT(N, R)                                                                                  \
    asm volatile("s_waitcnt lgkmcnt(" #N ")"                                                                \
                 : "+v"(R[0]), "+v"(R[1]), "+v"(R[2]), "+v"(R[3]), "+v"(R[4]), "+v"(R[5]), "+v"(R[6]), "+v"(R[7]))

__device__ __forceinline__ void fold_add_v(float& s, const fold_v4 (&R)[FOLD_B]) {
#pragma unroll
    for (int g = 0; g < FOLD_B; ++g) {
        s = s + R[g].x;
        s = s + R[g].y;
        s = s + R[g].z;
        s = s + R[g].w;
    }
}

__device__ __forceinline__ void fold_pass(float& s, uint32_t ad) {
    constexpr int BB = FOLD_B * CPW * 16;   // bytes between batches
    fold_v4 A[FOLD_B], B[FOLD_B];
    fold_issue_batch<0>(A, ad);
    fold_issue_batch<BB>(B, ad);
    AT_FOLD_WAIT(8, A);
    fold_add_v(s, A);
    fold_issue_batch<2 * BB>(A, ad);
    AT_FOLD_WAIT(8, B);
    fold_add_v(s, B);
    fold_issue_batch<3 * BB>(B, ad);
    AT_FOLD_WAIT(8, A);
    fold_add_v(s, A);
    AT_FOLD_WAIT(0, B);
    fold_add_v(s, B);
}
#undef AT_FOLD_WAIT

// The leaf values of chain block c0 for fold pass p (groups p*FOLD_P ..,
// one contiguous stretch of FOLD_P * CPW float4) moved by eight 1 KB
// direct-to-LDS loads of the calling wave into ring buffer p % FOLD_R1, so
// that entry g * CPW + j holds group g of chain c0 + j.  Past the last
// group the loads repeat the last float4 (never folded).
__device__ __forceinline__ void ring_issue_buf(const float4* __restrict__ blk, int last, float4* ring, int p, int b,
                                               int lane) {
    float4* buf = ring + b * (FOLD_P * CPW);
#pragma unroll
    for (int i = 0; i < FOLD_P * CPW / 64; ++i) {
        int idx = p * (FOLD_P * CPW) + i * 64 + lane;
        idx = idx < last ? idx : last;
        // non-temporal (cache policy 2): V is read once
        __builtin_amdgcn_global_load_lds(blk + idx, buf + i * 64, 16, 0, 2);
    }
}

__device__ __forceinline__ void ring_issue(const float4* __restrict__ blk, int last, float4* ring, int p, int lane) {
    ring_issue_buf(blk, last, ring, p, p % FOLD_R1, lane);
}

// Wait until at most `later` passes of this wave's ring moves are
// outstanding (the moves of older passes, and every older load, have
// landed).
#define AT_VM_WAIT(K) asm volatile("s_waitcnt vmcnt(" #K ")" ::: "memory")
__device__ __forceinline__ void ring_wait(int later) {
    static_assert(FOLD_P * CPW / 64 == 8 && FOLD_R1 <= 6 && FOLD_R2 <= 6,
                  "the waits below count eight moves per pass, at most five passes");
    switch (later) {
        case 0: AT_VM_WAIT(0); break;
        case 1: AT_VM_WAIT(8); break;
        case 2: AT_VM_WAIT(16); break;
        case 3: AT_VM_WAIT(24); break;
        case 4: AT_VM_WAIT(32); break;
        default: AT_VM_WAIT(40); break;
    }
}
#undef AT_VM_WAIT

// Groups (of four trees) in pass p of a model with `groups` groups.
__device__ __forceinline__ int pass_groups(int groups, int p) {
    return groups - p * FOLD_P < FOLD_P ? groups - p * FOLD_P : FOLD_P;
}

// One pass from the ring at src (the lane's column): ng groups, the last of
// them holding r trees when r > 0, added in tree order.
__device__ __forceinline__ void fold_pass_any(float& s, const float4* src, int ng, int r) {
    const int full = r ? ng - 1 : ng;
    int g = 0;
    if (full == FOLD_P) {
        fold_pass(s, lds_byte_address(src));
        g = FOLD_P;
    }
    for (; g + FOLD_B <= full; g += FOLD_B) {
        float4 A[FOLD_B];
        fold_load(A, src + g * CPW);
        fold_add(s, A);
    }
    for (; g < full; ++g) {
        const float4 q = src[g * CPW];
        s = s + q.x;
        s = s + q.y;
        s = s + q.z;
        s = s + q.w;
    }
    if (r) {
        const float4 q = src[full * CPW];
        s = s + q.x;
        if (r > 1) s = s + q.y;
        if (r > 2) s = s + q.z;
    }
}

// A full pass of each of two models (their ring buffers at LDS byte
// addresses ag and al), in batches of four groups of each, two register
// sets deep; the adds of the two sums alternate, so that each dependent add
// has the other sum's add beside it.
template <int OFF>
__device__ __forceinline__ void fold_issue_pair(fold_v4 (&R)[FOLD_B], uint32_t ag, uint32_t al) {
#define AT_FOLD_READ2(G, AD, O) \
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(R[G]) : "v"(AD), "i"(OFF + (O) * CPW * 16))
    AT_FOLD_READ2(0, ag, 0);
    AT_FOLD_READ2(1, ag, 1);
    AT_FOLD_READ2(2, ag, 2);
    AT_FOLD_READ2(3, ag, 3);
    AT_FOLD_READ2(4, al, 0);
    AT_FOLD_READ2(5, al, 1);
    AT_FOLD_READ2(6, al, 2);
    AT_FOLD_READ2(7, al, 3);
#undef AT_FOLD_READ2
}

__device__ __forceinline__ void fold_add_pair(float& sg, float& sl, const fold_v4 (&R)[FOLD_B]) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        sg = sg + R[g].x;
        sl = sl + R[4 + g].x;
        sg = sg + R[g].y;
        sl = sl + R[4 + g].y;
        sg = sg + R[g].z;
        sl = sl + R[4 + g].z;
        sg = sg + R[g].w;
        sl = sl + R[4 + g].w;
    }
}

#define AT_FOLD_WAIT2(N, R)                                                                                 \
    asm volatile("s_waitcnt lgkmcnt(" #N ")"                                                                \
                 : "+v"(R[0]), "+v"(R[1]), "+v"(R[2]), "+v"(R[3]), "+v"(R[4]), "+v"(R[5]), "+v"(R[6]), "+v"(R[7]))

__device__ __forceinline__ void fold_pass2(float& sg, uint32_t ag, float& sl, uint32_t al) {
    constexpr int BB = 4 * CPW * 16;   // bytes between batches of four groups
    static_assert(FOLD_P == 8 * 4, "a pass is eight batches of four groups");
    fold_v4 A[FOLD_B], B[FOLD_B];
    fold_issue_pair<0>(A, ag, al);
    fold_issue_pair<BB>(B, ag, al);
    AT_FOLD_WAIT2(8, A);
    fold_add_pair(sg, sl, A);
    fold_issue_pair<2 * BB>(A, ag, al);
    AT_FOLD_WAIT2(8, B);
    fold_add_pair(sg, sl, B);
    fold_issue_pair<3 * BB>(B, ag, al);
    AT_FOLD_WAIT2(8, A);
    fold_add_pair(sg, sl, A);
    fold_issue_pair<4 * BB>(A, ag, al);
    AT_FOLD_WAIT2(8, B);
    fold_add_pair(sg, sl, B);
    fold_issue_pair<5 * BB>(B, ag, al);
    AT_FOLD_WAIT2(8, A);
    fold_add_pair(sg, sl, A);
    fold_issue_pair<6 * BB>(A, ag, al);
    AT_FOLD_WAIT2(8, B);
    fold_add_pair(sg, sl, B);
    fold_issue_pair<7 * BB>(B, ag, al);
    AT_FOLD_WAIT2(8, A);
    fold_add_pair(sg, sl, A);
    AT_FOLD_WAIT2(0, B);
    fold_add_pair(sg, sl, B);
}
#undef AT_FOLD_WAIT2

// Score of the pending candidates of chain block c0 from one model's leaf
// values V (T trees): lane j < nc of the calling wave adds its chain's
// values in tree order (fp32, from +0.0f).  The wave alone moves the values
// into the LDS ring, FOLD_R1 passes ahead, so no other wave takes part.
// A pass's buffer is refilled at the start of the next pass, after its
// reads have completed.
__device__ __forceinline__ float fold_wave(const float* __restrict__ V, int T, int64_t c0, int nc, float4* ring,
                                           int lane) {
    const int groups = (T + 3) >> 2;
    const int npass = (groups + FOLD_P - 1) / FOLD_P;
    const float4* blk = reinterpret_cast<const float4*>(V) + (c0 >> 4) * (int64_t)groups * CPW;
    const int last = groups * CPW - 1;
    int issued = 0;
    for (; issued < FOLD_R1 - 1 && issued < npass; ++issued) ring_issue(blk, last, ring, issued, lane);
    float s = 0.0f;
    for (int p = 0; p < npass; ++p) {
        if (issued < npass) {
            ring_issue(blk, last, ring, issued, lane);
            ++issued;
        }
        ring_wait(issued - 1 - p);
        if (lane < nc) {
            const float4* src = ring + (p % FOLD_R1) * (FOLD_P * CPW) + lane;
            fold_pass_any(s, src, pass_groups(groups, p), (p == npass - 1) ? (T & 3) : 0);
        }
    }
    return s;
}

// Eq. 4: both models' scores, each its own fold in tree order from +0.0f.
// The two leaf-value arrays go through the one ring pass by pass in turn
// (pass m / 2 of the global model, then of the local one, while both have
// passes; then the longer one's last passes), and a pair of full passes is
// added with the two chains of dependent adds interleaved.
__device__ __forceinline__ void fold_wave2(const float* __restrict__ Vg, int Tg, const float* __restrict__ Vl, int Tl,
                                           int64_t c0, int nc, float4* ring, int lane, float& sg, float& sl) {
    const int gg = (Tg + 3) >> 2, gl = (Tl + 3) >> 2;
    const int npg = (gg + FOLD_P - 1) / FOLD_P, npl = (gl + FOLD_P - 1) / FOLD_P;
    const float4* bg = reinterpret_cast<const float4*>(Vg) + (c0 >> 4) * (int64_t)gg * CPW;
    const float4* bl = reinterpret_cast<const float4*>(Vl) + (c0 >> 4) * (int64_t)gl * CPW;
    const int pmin = npg < npl ? npg : npl, total = npg + npl;
    auto pass_of = [&](int m, bool& glob) -> int {
        if (m < 2 * pmin) {
            glob = (m & 1) == 0;
            return m >> 1;
        }
        glob = npg > npl;
        return m - pmin;
    };
    auto issue = [&](int m) {
        bool glob;
        const int p = pass_of(m, glob);
        ring_issue_buf(glob ? bg : bl, (glob ? gg : gl) * CPW - 1, ring, p, m % FOLD_R2, lane);
    };
    int issued = 0;
    for (; issued < FOLD_R2 - 1 && issued < total; ++issued) issue(issued);
    sg = 0.0f;
    sl = 0.0f;
    for (int m = 0; m < total;) {
        const bool pair = m < 2 * pmin;
        const int use = pair ? 2 : 1;
        // a pass's buffer is free once the pass FOLD_R2 before it was added
        for (; issued < total && issued < m + FOLD_R2; ++issued) issue(issued);
        ring_wait(issued - m - use);
        if (lane < nc) {
            if (pair) {
                const int p = m >> 1;
                const float4* srcg = ring + (m % FOLD_R2) * (FOLD_P * CPW) + lane;
                const float4* srcl = ring + ((m + 1) % FOLD_R2) * (FOLD_P * CPW) + lane;
                const int ngg = pass_groups(gg, p), ngl = pass_groups(gl, p);
                const int rg = (p == npg - 1) ? (Tg & 3) : 0, rl = (p == npl - 1) ? (Tl & 3) : 0;
                if (ngg == FOLD_P && ngl == FOLD_P && rg == 0 && rl == 0) {
                    fold_pass2(sg, lds_byte_address(srcg), sl, lds_byte_address(srcl));
                } else {
                    fold_pass_any(sg, srcg, ngg, rg);
                    fold_pass_any(sl, srcl, ngl, rl);
                }
            } else {
                bool glob;
                const int p = pass_of(m, glob);
                const float4* src = ring + (m % FOLD_R2) * (FOLD_P * CPW) + lane;
                if (glob)
                    fold_pass_any(sg, src, pass_groups(gg, p), (p == npg - 1) ? (Tg & 3) : 0);
                else
                    fold_pass_any(sl, src, pass_groups(gl, p), (p == npl - 1) ? (Tl & 3) : 0);
            }
        }
        m += use;
    }
}

// The first configuration of a chain: each knob uniform over its values,
// Philox block (chain, 0, 1, j / 4) word j % 4.
__device__ __forceinline__ void init_draw(const SpaceDesc& sd, uint32_t k0, uint32_t k1, uint32_t gchain,
                                          uint32_t (&nx)[MAX_KNOBS]) {
    U4 r{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) {
        if ((j & 3) == 0) r = philox(k0, k1, U4{gchain, 0u, 1u, (uint32_t)(j >> 2)});
        const uint32_t word = (j & 3) == 0 ? r.x : (j & 3) == 1 ? r.y : (j & 3) == 2 ? r.z : r.w;
        nx[j] = (j < sd.n_knobs) ? uniform_below(word, sd.knob_size[j]) : 0u;
    }
}

// The move of step `step` from configuration kv: one knob, uniform among
// those with two or more values, goes to a uniformly chosen other value;
// Philox block (chain, step, 0, 0).  The block does not depend on kv, so
// the moves from the two possible states of a step draw the same numbers.
__device__ __forceinline__ void step_move(const SpaceDesc& sd, uint32_t k0, uint32_t k1, uint32_t gchain,
                                          uint32_t step, const uint32_t (&kv)[MAX_KNOBS], uint32_t (&nx)[MAX_KNOBS]) {
    const U4 r = philox(k0, k1, U4{gchain, step, 0u, 0u});
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) nx[j] = kv[j];
    if (sd.n_mut > 0) {
        const int jm = sd.mut[uniform_below(r.x, (uint32_t)sd.n_mut)];
        uint32_t old = 0, size = 2;
#pragma unroll
        for (int j = 0; j < MAX_KNOBS; ++j)
            if (j == jm) {
                old = kv[j];
                size = sd.knob_size[j];
            }
        uint32_t nv = uniform_below(r.y, size - 1u);
        if (nv >= old) nv += 1u;
#pragma unroll
        for (int j = 0; j < MAX_KNOBS; ++j)
            if (j == jm) nx[j] = nv;
    }
}

// Loop l's eleven loop-context features of configuration nx into row[l *
// 11 ..], and bitlen(top-down product) into td[l] when asked for.
template <int TMPL>
__device__ __forceinline__ void row_features(const SpaceDesc& sd, const uint64_t* facp, const uint32_t (&nx)[MAX_KNOBS],
                                             int l, bool want_td, uint8_t* row, uint8_t* td) {
    uint32_t fac[6][4];
    gather_factors<TMPL>(sd, facp, nx, fac);
    uint32_t f[11], t = 0u;
    loop_features<TMPL>(sd, fac, ann_knobs_of<TMPL>(sd, nx), l, f, want_td ? &t : nullptr);
#pragma unroll
    for (int i = 0; i < 11; ++i) row[l * 11 + i] = (uint8_t)f[i];
    td[l] = (uint8_t)t;
}

__device__ __forceinline__ uint32_t pack_pair(const uint32_t (&nx)[MAX_KNOBS], int j) {
    return nx[2 * j] | (nx[2 * j + 1] << 16);
}

__device__ __forceinline__ void unpack_pairs(const uint32_t* w, uint32_t (&nx)[MAX_KNOBS]) {
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) nx[j] = (w[j >> 1] >> (16 * (j & 1))) & 0xffffu;
}

// Per-chain record of the chain kernel, shared through LDS.
struct TpRec {
    uint64_t cfg;                       // the pending candidate's configuration index
    float score;
    uint32_t count;                     // best list: entries, k-th entry
    float kth_score;
    uint32_t qual;
    uint64_t kth_cfg;
    uint32_t nx[2][MAX_KNOBS / 2];      // next candidate after an accept [0] or a reject [1]
};

// One annealing step of CPW chains (see the top of this file).  With a
// pending candidate, wave 0 folds its score while waves 1-3 bring the best
// lists into LDS and build, for every chain, both candidates that can come
// next (a move from the pending candidate if it is accepted, from the
// current configuration if not) and the loop-context features of both;
// once the score is known the owner lanes (wave 0, lane j: chain c0 + j)
// offer the candidate to the best list, take the Metropolis decision and
// the rows of the candidate that follows go out.
template <int TMPL, int CHAIN_WG>
__global__ __launch_bounds__(CHAIN_WG) void k_chain(ChainArgs a) {
    using N = Nest<TMPL>;
    constexpr int L = N::L;
    constexpr int Q = (N::F + 3) / 4;
    constexpr int RS = Q * 4 + 4;                 // feature row stride (bytes) in LDS
    // dynamic LDS: the fold ring, then the chains' best lists [CPW][topk]
    extern __shared__ float4 ring[];
    __shared__ TpRec rec[CPW];
    __shared__ __attribute__((aligned(16))) uint8_t frow[2][CPW][RS];
    __shared__ uint8_t tdrow[2][CPW][16];
    __shared__ __attribute__((aligned(16))) uint8_t s_img[STAGE_MAX_BYTES];
    __shared__ __attribute__((aligned(16))) uint16_t s_kv[2][CPW][MAX_KNOBS];   // current, pending knobs
    __shared__ uint32_t s_sel[CPW];
    __shared__ uint32_t s_any;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t c0 = (int64_t)blockIdx.x * CPW;
    const int nc = (a.n - c0 < CPW) ? (int)(a.n - c0) : CPW;
    const bool owner = tid < nc;                 // lanes of wave 0 that own a chain
    const int64_t c = c0 + (owner ? tid : 0);
    const int k = a.topk;
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    // group of 16 lanes per chain for the best-list offer and the features
    const int gj = tid >> 4, gr = tid & 15;
    const uint64_t gmask = 0xffffull << (16 * (gj & 3));
    const bool gvalid = gj < nc;
    at_entry* lists = reinterpret_cast<at_entry*>(ring + ring_bytes(a.Vg != nullptr) / 16);

    // The workgroup's space: when all its chains share one space whose image
    // fits, the image (descriptor with rebased split offsets, then the split
    // factors) moves straight into LDS; otherwise each lane reads its own
    // chain's space from global memory.
    const int ws = a.n_spaces == 1 ? a.stage_single : a.wg_space[blockIdx.x];
    const bool staged = ws >= 0;
    const SpaceDesc* s_desc = reinterpret_cast<const SpaceDesc*>(s_img);
    const uint64_t* facp = staged ? reinterpret_cast<const uint64_t*>(s_img + STAGE_DESC_BYTES) : a.factors;
    auto desc_of = [&](int j) -> const SpaceDesc& {
        return staged ? *s_desc : a.descs[space_of(a.offsets, a.n_spaces, c0 + j)];
    };
    auto copy_image = [&](int first, int stride) {
        const uint8_t* src = a.stage + (int64_t)ws * a.stage_stride + lane * 16;
        for (int off = first * 1024; off < a.stage_stride; off += stride * 1024)
            __builtin_amdgcn_global_load_lds(src + off, s_img + off, 16, 0, 0);
    };

    // per-chain state of the owner lanes, in flight while the score is
    // folded.  Every lane loads from valid addresses (c is chain c0 for lanes
    // that own no chain; the threshold is read from the scores when there is
    // none), so no branch joins the loaded values: a join would wait for them.
    uint2 kraw[3], craw[3];
    load_knob_words(a.knobs, c, kraw);
    load_knob_words(a.cand, c, craw);
    ChainMeta m = a.meta[c];
    const float cur_s = a.cur_score[c];
    const float* thr_b = a.fin == FIN_STEP ? a.thr : a.cur_score;
    int64_t thr_i = a.fin == FIN_STEP ? c * a.steps + a.fin_step : c;
    asm volatile("" : "+v"(thr_i));   // one load from either table (not two loads and a join)
    const float thr_v = thr_b[thr_i];
    // tile-layout words of the packed rows this thread writes at the end
    // (quads (tid + m * CHAIN_WG) / 16, clamped to the last so that every
    // lane loads)
    constexpr int PACK_ITERS = (CPW * Q + CHAIN_WG - 1) / CHAIN_WG;
    uint32_t src4[PACK_ITERS];
#pragma unroll
    for (int m = 0; m < PACK_ITERS; ++m) src4[m] = 0u;
    if (!a.fident) {
#pragma unroll
        for (int m = 0; m < PACK_ITERS; ++m) {
            const int q = (tid + m * CHAIN_WG) >> 4;
            src4[m] = *reinterpret_cast<const uint32_t*>(a.fsrc + 4 * (q < a.fq ? q : a.fq - 1));
        }
    }

    if (a.fin == FIN_NONE) {
        // No pending candidate: the first draw of fresh chains, or a move
        // from the current configurations, or only the best lists' copy.
        if (a.best) {
            for (int idx = tid; idx < nc * k; idx += CHAIN_WG) a.best[c0 * k + idx] = a.top[c0 * k + idx];
        }
        if (a.draw == DRAW_NONE) return;
        if (staged) copy_image(wave, CHAIN_WG / 64);
        asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
        if (owner) {
            const SpaceDesc& sd = desc_of(tid);
            const uint32_t gchain = (uint32_t)(a.chain0 + (uint64_t)c);
            uint32_t nx[MAX_KNOBS];
            if (a.draw == DRAW_INIT) {
                init_draw(sd, k0, k1, gchain, nx);
            } else {
                uint32_t cur[MAX_KNOBS];
                unpack_knobs(kraw, cur);
                step_move(sd, k0, k1, gchain, a.draw_step, cur, nx);
            }
            store_knobs(a.cand, c, nx);
#pragma unroll
            for (int j = 0; j < MAX_KNOBS / 2; ++j) rec[tid].nx[0][j] = pack_pair(nx, j);
            s_sel[tid] = 0u;
        }
        lds_barrier();
        // lane gr of group gj: loop gr of chain gj's candidate
        if (gvalid && gr < L) {
            uint32_t nx[MAX_KNOBS];
            unpack_pairs(rec[gj].nx[0], nx);
            row_features<TMPL>(desc_of(gj), facp, nx, gr, a.Fr != nullptr, frow[0][gj], tdrow[0][gj]);
        }
        lds_barrier();
    } else {
        float s = 0.0f;
        if (wave == 0) {
            // the fold is a chain of dependent adds: its wave goes first
            // whenever it can issue, ahead of the candidate building
            __builtin_amdgcn_s_setprio(3);
            // Eq. 4: each model's prediction is its own fold from +0.0f; the
            // sum adds the global one first
            if (a.Vg) {
                float sg, sl;
                fold_wave2(a.Vg, a.Tg, a.V, a.T, c0, nc, ring, lane, sg, sl);
                s = sg + sl;
            } else {
                s = fold_wave(a.V, a.T, c0, nc, ring, lane);
            }
            __builtin_amdgcn_s_setprio(0);
        } else {
            // waves 1-3: each copies the whole space image and the chains'
            // knobs (identical bytes, so the copies may overlap) and waits
            // for its own moves only; the best lists are shared out
            if (staged) copy_image(0, 1);
            {
                const int nb = nc * MAX_KNOBS * 2;           // bytes of one knob array
                const uint8_t* kp = reinterpret_cast<const uint8_t*>(a.knobs + c0 * MAX_KNOBS);
                const uint8_t* cp = reinterpret_cast<const uint8_t*>(a.cand + c0 * MAX_KNOBS);
                uint8_t* d = reinterpret_cast<uint8_t*>(&s_kv[0][0][0]);
                constexpr int KB = CPW * MAX_KNOBS * 2;      // LDS bytes of one knob array
                static_assert(2 * KB == 3 * 256, "three dword moves of 64 lanes");
#pragma unroll
                for (int i = 0; i < 3; ++i) {
                    const int byte = i * 256 + lane * 4;     // of the two arrays, current first
                    const int arr = byte >= KB ? 1 : 0, off = byte - arr * KB;
                    if (off < nb) __builtin_amdgcn_global_load_lds((arr ? cp : kp) + off, d + i * 256, 4, 0, 0);
                }
            }
            if (a.fin == FIN_STEP) {
                const at_entry* src = a.top + c0 * k;
                const int total = nc * k;
                for (int ins = wave - 1; ins * 64 < total; ins += CHAIN_WG / 64 - 1) {
                    const int e = ins * 64 + lane;
                    if (e < total) __builtin_amdgcn_global_load_lds(src + e, lists + ins * 64, 16, 0, 0);
                }
            } else {
                // an initial list is empty
                for (int e = tid - 64; e < nc * k; e += CHAIN_WG - 64) {
                    at_entry z;
                    z.cfg = 0;
                    z.score = 0.0f;
                    z.flag = 0u;
                    lists[e] = z;
                }
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            // the pending candidates' configuration indices
            const int t0 = tid - 64;
            if (t0 < nc) {
                const SpaceDesc& sd = desc_of(t0);
                uint64_t cfg = 0;
#pragma unroll
                for (int j = 0; j < MAX_KNOBS; ++j)
                    if (j < sd.n_knobs) cfg += (uint64_t)s_kv[1][t0][j] * sd.radix[j];
                rec[t0].cfg = cfg;
            }
            // both next candidates of every chain and their loop features:
            // task t is loop t % L of outcome (t / L) & 1 of chain t / (2L)
            // (an initial candidate is always accepted: no reject outcome)
            if (a.draw == DRAW_PROPOSE) {
                // the moves first, lane i < 2 nc of every building wave making
                // the move of chain i / 2 from state i & 1 into the wave's own
                // rows (the same values in every wave, so none waits for
                // another), then the loop tasks from those rows
                __shared__ uint32_t s_mv[CHAIN_WG / 64 - 1][2 * CPW][MAX_KNOBS / 2];
                uint32_t(*mv)[MAX_KNOBS / 2] = s_mv[wave - 1];
                if (lane < 2 * nc && !((lane & 1) == 1 && a.fin == FIN_INIT)) {
                    const int j = lane >> 1, o = lane & 1;
                    const SpaceDesc& sd = desc_of(j);
                    uint32_t base[MAX_KNOBS], nx[MAX_KNOBS];
#pragma unroll
                    for (int i = 0; i < MAX_KNOBS; ++i) base[i] = s_kv[o ^ 1][j][i];
                    step_move(sd, k0, k1, (uint32_t)(a.chain0 + (uint64_t)(c0 + j)), a.draw_step, base, nx);
#pragma unroll
                    for (int i = 0; i < MAX_KNOBS / 2; ++i) {
                        mv[lane][i] = pack_pair(nx, i);
                        if (wave == 1) rec[j].nx[o][i] = pack_pair(nx, i);
                    }
                }
                __builtin_amdgcn_s_waitcnt(0xc07f);
                __builtin_amdgcn_wave_barrier();
                for (int t = t0; t < nc * 2 * L; t += CHAIN_WG - 64) {
                    const int l = t % L, jo = t / L, j = jo >> 1, o = jo & 1;
                    if (o == 1 && a.fin == FIN_INIT) continue;
                    uint32_t nx[MAX_KNOBS];
                    unpack_pairs(mv[jo], nx);
                    row_features<TMPL>(desc_of(j), facp, nx, l, a.Fr != nullptr, frow[o][j], tdrow[o][j]);
                }
            }
            if (a.pf_trees) {
                // the next tree launch copies its trees from the L2: chain
                // workgroup b takes half of the trees of tree workgroup
                // 8 * (b / 16) + b % 8, which runs on the same XCD when
                // workgroups go round the eight XCDs in turn (a wrong guess
                // only warms another XCD's L2)
                const int b = (int)blockIdx.x;
                const int tw = 8 * (b / 16) + b % 8, half = (b / 8) & 1;
                const int per = a.pf_tpw / 2 > 0 ? a.pf_tpw / 2 : 1;
                const int first = tw * a.pf_tpw + half * per;
                int cnt = a.pf_ntrees - first < per ? a.pf_ntrees - first : per;
                if (half == 1 && a.pf_tpw == 1) cnt = 0;
                if (cnt > 0) {
                    const int64_t bytes = (int64_t)cnt * a.pf_tree_bytes;
                    const uint8_t* src = a.pf_trees + (int64_t)first * a.pf_tree_bytes;
                    // plain loads, all in flight before one wait: each lane
                    // takes 16 bytes of every 1 KB line its wave covers (at most
                    // PF_LINES lines a wave), from a valid address on every
                    // lane, the values folded into one that is kept
                    constexpr int PF_LINES = 12;
                    const int nbw = CHAIN_WG / 64 - 1;
                    uint32_t keep = 0u;
                    uint4 v[PF_LINES];
#pragma unroll
                    for (int u = 0; u < PF_LINES; ++u) {
                        int64_t off = ((int64_t)u * nbw + (wave - 1)) * 1024 + lane * 16;
                        off = off < bytes ? off : bytes - 16;
                        v[u] = *reinterpret_cast<const uint4*>(src + off);
                    }
#pragma unroll
                    for (int u = 0; u < PF_LINES; ++u) keep ^= v[u].x;
                    asm volatile("" ::"v"(keep));
                }
            }
        }
        // score known (wave 0), candidates built (waves 1-3)
        lds_barrier();

        // owner lanes: qualification for the best list, the Metropolis
        // decision, the chain's state
        int qual = 0;
        bool acc = true;
        if (owner) {
            if (a.fin != FIN_STEP) {
                // a fresh chain: empty best list
                m.count = 0;
                m.kth_score = 0.0f;
                m.kth_cfg = 0;
            }
            TpRec& R = rec[tid];
            const uint64_t cfg = R.cfg;
            qual = (a.fin == FIN_INIT || (int)m.count < k || precedes(s, cfg, m.kth_score, m.kth_cfg)) ? 1 : 0;
            R.score = s;
            R.count = m.count;
            R.kth_score = m.kth_score;
            R.kth_cfg = m.kth_cfg;
            R.qual = (uint32_t)qual;
            if (a.fin == FIN_STEP) {
                const float delta = s - cur_s;
                acc = delta >= thr_v;
                if (a.trace) {
                    at_entry t;
                    t.cfg = cfg;
                    t.score = s;
                    t.flag = acc ? 1u : 0u;
                    a.trace[c * a.steps + a.fin_step] = t;
                }
            }
            if (acc) {
                reinterpret_cast<uint2*>(a.knobs)[3 * c] = craw[0];
                reinterpret_cast<uint2*>(a.knobs)[3 * c + 1] = craw[1];
                reinterpret_cast<uint2*>(a.knobs)[3 * c + 2] = craw[2];
                a.cur_score[c] = s;
            }
            const int o = acc ? 0 : 1;
            s_sel[tid] = (uint32_t)o;
            if (a.draw == DRAW_PROPOSE) {
                uint2* w = reinterpret_cast<uint2*>(a.cand) + 3 * c;
                w[0] = make_uint2(R.nx[o][0], R.nx[o][1]);
                w[1] = make_uint2(R.nx[o][2], R.nx[o][3]);
                w[2] = make_uint2(R.nx[o][4], R.nx[o][5]);
            }
        } else if (tid < CPW) {
            rec[tid].qual = 0;
        }
        if (wave == 0) {
            const uint64_t q = __ballot(qual);
            if (tid == 0) s_any = q != 0 ? 1u : 0u;
        }
        // the barriers from here on order LDS only: a full __syncthreads
        // would also wait for this workgroup's global stores (best lists,
        // trace, state) to drain
        lds_barrier();

        // best lists: the chain's group of 16 lanes inserts the candidate
        // into its list in LDS when it qualifies, each lane writing the
        // entries it changes (and the new count and k-th entry) to global
        // memory as well.  Skipped when no chain qualifies.
        if (s_any) {
            const int64_t cg = c0 + (gvalid ? gj : 0);
            group_offer(lists + gj * k, rec[gj], k, gr, gmask, gvalid && rec[gj].qual != 0, a.top + cg * k,
                        a.meta + cg);
        }
        if (a.best) {
            lds_barrier();
            for (int idx = tid; idx < nc * k; idx += CHAIN_WG) a.best[c0 * k + idx] = lists[idx];
        }
        if (a.draw == DRAW_NONE) return;
    }

    // the rows of each chain's next candidate: outcome s_sel[j] (rows and
    // choices are in LDS since the last barrier)
    if (a.Fr) {
        // context relation features of the candidate (Section 4): output
        // o = [pair][buffer b][t - 1] is the largest value over the loops
        // whose touch count of b is below 2^t (bitlen(touch) <= t), the value
        // being bitlen(reuse ratio of b) for pair 0, bitlen(top-down) for
        // pair 1; 0 when no loop qualifies.  Lane gr of group gj makes
        // outputs gr, gr + 16, ...
        __shared__ __attribute__((aligned(16))) uint8_t rrow[CPW][REL_F];
        if (gvalid) {
            const uint8_t* fr = frow[s_sel[gj]][gj];
            const uint8_t* tr = tdrow[s_sel[gj]][gj];
#pragma unroll 1
            for (int o = gr; o < REL_F; o += 16) {
                const int pair = o / 96, b = (o >> 5) % 3;
                const uint32_t t = (uint32_t)(o & 31) + 1u;
                uint32_t v = 0u;
#pragma unroll
                for (int l = 0; l < L; ++l) {
                    const uint32_t bt = fr[l * 11 + 2 + 3 * b];
                    const uint32_t x = pair ? (uint32_t)tr[l] : (uint32_t)fr[l * 11 + 3 + 3 * b];
                    v = (bt <= t && x > v) ? x : v;
                }
                rrow[gj][o] = (uint8_t)v;
            }
        }
        lds_barrier();
        for (int idx = tid; idx < CPW * REL_Q; idx += CHAIN_WG) {
            const int q = idx >> 4, j = idx & (CPW - 1);
            if (j >= nc) continue;
            const uint32_t w = (*reinterpret_cast<const uint32_t*>(&rrow[j][4 * q]) << 2) | 0x03030303u;
            a.Fr[(int64_t)q * a.fg_stride + c0 + j] = w;
        }
    }
    // packed rows out in the tree kernel's tile layout (4x+3 per byte,
    // padding 0), consecutive lanes on consecutive chains
    // (a feature value x <= 63 makes (x << 2) | 3 stay within its byte)
#pragma unroll
    for (int m = 0; m < PACK_ITERS; ++m) {
        const int idx = tid + m * CHAIN_WG;
        const int q = idx >> 4, j = idx & (CPW - 1);
        if (q >= a.fq || j >= nc) continue;
        const uint8_t* row = frow[s_sel[j]][j];
        uint32_t w = 0u;
        if (a.fident) {
            constexpr uint32_t LAST = (N::F & 3) ? (1u << (8 * (N::F & 3))) - 1u : 0xffffffffu;
            w = (*reinterpret_cast<const uint32_t*>(row + 4 * q) << 2) | 0x03030303u;
            if (q == Q - 1) w &= LAST;
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t f = (src4[m] >> (8 * i)) & 0xffu;
                if (f != 0xffu) w |= (((uint32_t)row[f] << 2) | 3u) << (8 * i);
            }
        }
        a.Fg[(int64_t)q * a.fg_stride + c0 + j] = w;
    }
}

// ---------------------------------------------------------------------------
// Tree kernel.  A workgroup holds the pointer form of its trees in LDS and
// walks them for every chain.  Each wave owns a feature tile of 64 chains in
// a slot of SLOT bytes (a power of two) at wave * SLOT: byte (p & 3) of
// dword (p >> 2) * 64 + lane holds 4x+3 for the value x of the feature at
// tile position p, so lanes read distinct banks whatever features they ask
// for, and the tile byte address of position p is (node & mask) | (wave *
// SLOT + 4 * lane) for a node of that feature, mask = 3 | (SLOT - 1) & ~0xff.
// A tile holds the space's varying loop-context features only: a node on a
// feature that is constant over the space was settled when the trees were
// relocated (both children made the one it reaches).
// With 4x+3 in the tile, x >= thr is (4x+3) >= (low byte of the node) for
// x, thr <= 63.  Tiles are private to their wave, so the walk loop needs no
// barrier; tree blocks go into the gaps after the tiles.
// ---------------------------------------------------------------------------
constexpr int TREES_MAX = 16;          // trees per workgroup
constexpr int TREE_WAVES_MAX = 16;

struct TreeArgs {
    const uint32_t* words32;   // pointer form relocated for toff (k_reloc)
    int n_trees;
    int tpw;                   // trees per workgroup
    const uint32_t* Fg;        // [Q][fg_stride] packed features (4x+3 per byte)
    int64_t fg_stride;         // n rounded up to 64 chains
    int64_t n;
    float* V;
    int slices;                // chain slices per tree group
    int slice_blocks;          // 64-chain blocks per slice
    int q;                     // quads (4 features) per chain in a tile
    uint32_t slot;             // bytes per wave's tile slot
    uint32_t counter;          // LDS byte offset of the block counter
    uint32_t mask;             // node bits of a tile address: 3 | (slot - 1) & ~0xff
    // LDS dword offsets of tree i's node block (low half) and leaf block (high half)
    uint32_t toff[TREES_MAX];
};

// Tree walks over the pointer form.  A node is 32 bits: its compact node in
// the low half and its children's LDS address / 4 in the high half, so the
// children's slot is at node >> 14 (bits 14-15 of a compact node are zero).
// A level reads the node's feature byte from the tile and its children's
// 8-byte slot, then keeps the right child when (node & 0xff) <= x4.  After
// DEPTH levels the kept word is the leaf value.  nb[g] is the LDS address
// of tree g's node block (the root is its first word).

// Plain walk of G trees (any DEPTH).
template <int DEPTH, int G>
__device__ __forceinline__ void walk_plain(const uint8_t* __restrict__ L, const uint32_t (&nb)[G], uint32_t fb,
                                           uint32_t mask, uint32_t (&out)[G]) {
    uint32_t node[G];
#pragma unroll
    for (int g = 0; g < G; ++g) node[g] = *reinterpret_cast<const uint32_t*>(L + nb[g]);
#pragma unroll
    for (int l = 0; l < DEPTH; ++l) {
        uint32_t x4[G];
        uint64_t pr[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            x4[g] = L[(node[g] & mask) | fb];
            pr[g] = *reinterpret_cast<const uint64_t*>(L + (node[g] >> 14));
        }
#pragma unroll
        for (int g = 0; g < G; ++g) node[g] = x4[g] >= (node[g] & 0xffu) ? (uint32_t)(pr[g] >> 32) : (uint32_t)pr[g];
    }
#pragma unroll
    for (int g = 0; g < G; ++g) out[g] = node[g];
}

// One level of four trees: right = (node & 0xff) <= x4 (the compiler does
// not form the byte compare from plain code), node = right ? hi : lo, then
// the next feature address (node & mask) | fb and slot address node >> 14.
// A VALU write of VCC is read two or more instructions later (gfx950 wait
// states): the first compare is followed by s_nop 1, the others by the
// previous tree's address instructions.
// Operands: 0-3 node, 4-7 feature address, 8-11 slot address, 12-15 x4,
// 16-19 lo, 20-23 hi, 24 mask, 25 fb.
#define AT_PLEVEL4_ASM                                                                                     \
    "v_cmp_le_u32_sdwa vcc, %0, %12 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32 %0, %16, %20, vcc\n\t"                                                                   \
    "v_cmp_le_u32_sdwa vcc, %1, %13 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %4, %0, %24, %25\n\t"                                                                    \
    "v_lshrrev_b32 %8, 14, %0\n\t"                                                                         \
    "v_cndmask_b32 %1, %17, %21, vcc\n\t"                                                                   \
    "v_cmp_le_u32_sdwa vcc, %2, %14 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %5, %1, %24, %25\n\t"                                                                    \
    "v_lshrrev_b32 %9, 14, %1\n\t"                                                                         \
    "v_cndmask_b32 %2, %18, %22, vcc\n\t"                                                                   \
    "v_cmp_le_u32_sdwa vcc, %3, %15 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %6, %2, %24, %25\n\t"                                                                    \
    "v_lshrrev_b32 %10, 14, %2\n\t"                                                                        \
    "v_cndmask_b32 %3, %19, %23, vcc\n\t"                                                                   \
    "v_and_or_b32 %7, %3, %24, %25\n\t"                                                                    \
    "v_lshrrev_b32 %11, 14, %3"

// The last level of four trees: the kept word is the leaf value.
// Operands: 0-3 node, 4-7 x4, 8-11 lo, 12-15 hi.
#define AT_PLAST4_ASM                                                                                      \
    "v_cmp_le_u32_sdwa vcc, %0, %4 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                     \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32 %0, %8, %12, vcc\n\t"                                                                    \
    "v_cmp_le_u32_sdwa vcc, %1, %5 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                     \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32 %1, %9, %13, vcc\n\t"                                                                    \
    "v_cmp_le_u32_sdwa vcc, %2, %6 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                     \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32 %2, %10, %14, vcc\n\t"                                                                   \
    "v_cmp_le_u32_sdwa vcc, %3, %7 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                     \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32 %3, %11, %15, vcc"

// Reads of one level for four trees: feature byte and children's slot.
// Operands: 0-3 x4, 4-7 slot (64-bit), 8-11 feature address, 12-15 slot
// address.
#define AT_PISSUE4_ASM                                                                                     \
    "ds_read_u8 %0, %8\n\t"                                                                                \
    "ds_read_b64 %4, %12\n\t"                                                                              \
    "ds_read_u8 %1, %9\n\t"                                                                                \
    "ds_read_b64 %5, %13\n\t"                                                                              \
    "ds_read_u8 %2, %10\n\t"                                                                               \
    "ds_read_b64 %6, %14\n\t"                                                                              \
    "ds_read_u8 %3, %11\n\t"                                                                               \
    "ds_read_b64 %7, %15"

// Eight trees as two software-pipelined groups of four (A = trees 0-3, B =
// 4-7).  A group's step waits for its own reads (LDS answers in issue
// order, so lgkmcnt(8) leaves just the other group's eight in flight),
// computes the level and at once issues the reads of its next level; the
// other group's reads are served meanwhile.  Reads live across asm
// statements: the wait is a statement of its own that takes the receiving
// registers as in-out operands, so whatever the compiler does with them
// comes after the wait.  The asm takes offsets into L as LDS addresses: L
// is the kernel's only LDS object, so it starts at LDS address 0 (the
// launcher checks that the kernel's static LDS is that array alone).
template <int DEPTH, bool ROOTS>
__device__ __forceinline__ void walk8_roll(const uint8_t* __restrict__ L, const uint32_t (&nb)[8], uint32_t fb,
                                           uint32_t mask, const uint32_t (&rnode)[8], const uint32_t (&rlo)[8],
                                           const uint32_t (&rhi)[8], uint32_t (&out)[8]) {
    uint32_t node[8], fa[8], pa[8], x4[8];
    uint64_t pr[8];
    int l0 = 0;
    if constexpr (ROOTS) {
        // roots and their children's slots are given: level 0 needs only
        // the feature bytes
        static_assert(DEPTH >= 2, "a level below the root");
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            node[g] = rnode[g];
            fa[g] = (rnode[g] & mask) | fb;
        }
#pragma unroll
        for (int h = 0; h < 8; h += 4)
            asm volatile("ds_read_u8 %0, %4\n\t"
                         "ds_read_u8 %1, %5\n\t"
                         "ds_read_u8 %2, %6\n\t"
                         "ds_read_u8 %3, %7"
                         : "=&v"(x4[h]), "=&v"(x4[h + 1]), "=&v"(x4[h + 2]), "=&v"(x4[h + 3])
                         : "v"(fa[h]), "v"(fa[h + 1]), "v"(fa[h + 2]), "v"(fa[h + 3])
                         : "memory");
#pragma unroll
        for (int h = 0; h < 8; h += 4) {
            // group A waits for its four reads (group B's four are behind
            // them), group B for its four (group A's next eight are behind)
            if (h == 0)
                asm volatile("s_waitcnt lgkmcnt(4)" : "+v"(x4[h]), "+v"(x4[h + 1]), "+v"(x4[h + 2]), "+v"(x4[h + 3]));
            else
                asm volatile("s_waitcnt lgkmcnt(8)" : "+v"(x4[h]), "+v"(x4[h + 1]), "+v"(x4[h + 2]), "+v"(x4[h + 3]));
            asm volatile(AT_PLEVEL4_ASM
                         : "+v"(node[h]), "+v"(node[h + 1]), "+v"(node[h + 2]), "+v"(node[h + 3]), "=&v"(fa[h]),
                           "=&v"(fa[h + 1]), "=&v"(fa[h + 2]), "=&v"(fa[h + 3]), "=&v"(pa[h]), "=&v"(pa[h + 1]),
                           "=&v"(pa[h + 2]), "=&v"(pa[h + 3])
                         : "v"(x4[h]), "v"(x4[h + 1]), "v"(x4[h + 2]), "v"(x4[h + 3]), "v"(rlo[h]), "v"(rlo[h + 1]),
                           "v"(rlo[h + 2]), "v"(rlo[h + 3]), "v"(rhi[h]), "v"(rhi[h + 1]), "v"(rhi[h + 2]),
                           "v"(rhi[h + 3]), "s"(mask), "v"(fb)
                         : "vcc");
            asm volatile(AT_PISSUE4_ASM
                         : "=&v"(x4[h]), "=&v"(x4[h + 1]), "=&v"(x4[h + 2]), "=&v"(x4[h + 3]), "=&v"(pr[h]),
                           "=&v"(pr[h + 1]), "=&v"(pr[h + 2]), "=&v"(pr[h + 3])
                         : "v"(fa[h]), "v"(fa[h + 1]), "v"(fa[h + 2]), "v"(fa[h + 3]), "v"(pa[h]), "v"(pa[h + 1]),
                           "v"(pa[h + 2]), "v"(pa[h + 3]));
        }
        l0 = 1;
    } else {
#pragma unroll
        for (int g = 0; g < 8; ++g) {
            node[g] = *reinterpret_cast<const uint32_t*>(L + nb[g]);
            fa[g] = (node[g] & mask) | fb;
            pa[g] = node[g] >> 14;
        }
#pragma unroll
        for (int h = 0; h < 8; h += 4)
            asm volatile(AT_PISSUE4_ASM
                         : "=&v"(x4[h]), "=&v"(x4[h + 1]), "=&v"(x4[h + 2]), "=&v"(x4[h + 3]), "=&v"(pr[h]),
                           "=&v"(pr[h + 1]), "=&v"(pr[h + 2]), "=&v"(pr[h + 3])
                         : "v"(fa[h]), "v"(fa[h + 1]), "v"(fa[h + 2]), "v"(fa[h + 3]), "v"(pa[h]), "v"(pa[h + 1]),
                           "v"(pa[h + 2]), "v"(pa[h + 3])
                         : "memory");
    }
#pragma unroll
    for (int l = 0; l + 1 < DEPTH; ++l) {
        if (l < l0) continue;
#pragma unroll
        for (int h = 0; h < 8; h += 4) {
            asm volatile("s_waitcnt lgkmcnt(8)"
                         : "+v"(x4[h]), "+v"(x4[h + 1]), "+v"(x4[h + 2]), "+v"(x4[h + 3]), "+v"(pr[h]),
                           "+v"(pr[h + 1]), "+v"(pr[h + 2]), "+v"(pr[h + 3]));
            asm volatile(AT_PLEVEL4_ASM
                         : "+v"(node[h]), "+v"(node[h + 1]), "+v"(node[h + 2]), "+v"(node[h + 3]), "=&v"(fa[h]),
                           "=&v"(fa[h + 1]), "=&v"(fa[h + 2]), "=&v"(fa[h + 3]), "=&v"(pa[h]), "=&v"(pa[h + 1]),
                           "=&v"(pa[h + 2]), "=&v"(pa[h + 3])
                         : "v"(x4[h]), "v"(x4[h + 1]), "v"(x4[h + 2]), "v"(x4[h + 3]), "v"((uint32_t)pr[h]),
                           "v"((uint32_t)pr[h + 1]), "v"((uint32_t)pr[h + 2]), "v"((uint32_t)pr[h + 3]),
                           "v"((uint32_t)(pr[h] >> 32)), "v"((uint32_t)(pr[h + 1] >> 32)),
                           "v"((uint32_t)(pr[h + 2] >> 32)), "v"((uint32_t)(pr[h + 3] >> 32)), "s"(mask), "v"(fb)
                         : "vcc");
            asm volatile(AT_PISSUE4_ASM
                         : "=&v"(x4[h]), "=&v"(x4[h + 1]), "=&v"(x4[h + 2]), "=&v"(x4[h + 3]), "=&v"(pr[h]),
                           "=&v"(pr[h + 1]), "=&v"(pr[h + 2]), "=&v"(pr[h + 3])
                         : "v"(fa[h]), "v"(fa[h + 1]), "v"(fa[h + 2]), "v"(fa[h + 3]), "v"(pa[h]), "v"(pa[h + 1]),
                           "v"(pa[h + 2]), "v"(pa[h + 3]));
        }
    }
#pragma unroll
    for (int h = 0; h < 8; h += 4) {
        if (h == 0)
            asm volatile("s_waitcnt lgkmcnt(8)"
                         : "+v"(x4[h]), "+v"(x4[h + 1]), "+v"(x4[h + 2]), "+v"(x4[h + 3]), "+v"(pr[h]),
                           "+v"(pr[h + 1]), "+v"(pr[h + 2]), "+v"(pr[h + 3]));
        else
            asm volatile("s_waitcnt lgkmcnt(0)"
                         : "+v"(x4[h]), "+v"(x4[h + 1]), "+v"(x4[h + 2]), "+v"(x4[h + 3]), "+v"(pr[h]),
                           "+v"(pr[h + 1]), "+v"(pr[h + 2]), "+v"(pr[h + 3]));
        asm volatile(AT_PLAST4_ASM
                     : "+v"(node[h]), "+v"(node[h + 1]), "+v"(node[h + 2]), "+v"(node[h + 3])
                     : "v"(x4[h]), "v"(x4[h + 1]), "v"(x4[h + 2]), "v"(x4[h + 3]), "v"((uint32_t)pr[h]),
                       "v"((uint32_t)pr[h + 1]), "v"((uint32_t)pr[h + 2]), "v"((uint32_t)pr[h + 3]),
                       "v"((uint32_t)(pr[h] >> 32)), "v"((uint32_t)(pr[h + 1] >> 32)),
                       "v"((uint32_t)(pr[h + 2] >> 32)), "v"((uint32_t)(pr[h + 3] >> 32))
                     : "vcc");
    }
#pragma unroll
    for (int g = 0; g < 8; ++g) out[g] = node[g];
}

template <int DEPTH, int G>
__device__ __forceinline__ void walk_vals(const uint8_t* __restrict__ L, const TreeArgs& a, int t, uint32_t fb,
                                          uint32_t (&v)[G]) {
    uint32_t nb[G];
#pragma unroll
    for (int g = 0; g < G; ++g) nb[g] = (a.toff[t + g] & 0xffffu) * 4u;
    if constexpr (G == 8) {
        const uint32_t none[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        walk8_roll<DEPTH, false>(L, nb, fb, a.mask, none, none, none, v);
    } else
        walk_plain<DEPTH, G>(L, nb, fb, a.mask, v);
}

// Leaf values go to V with non-temporal stores: each is read once, by the
// chain kernel, and the L2 is better spent on features and trees.
template <int G>
__device__ __forceinline__ void store_vals(const TreeArgs& a, int t_global, int64_t c, const uint32_t (&v)[G]) {
    const int groups = (a.n_trees + 3) >> 2;
    float* dst = a.V + v_index(c, t_global, groups);
    if (G >= 4 && (t_global & 3) == 0) {
#pragma unroll
        for (int h = 0; h + 4 <= G; h += 4) {
            typedef float f4v __attribute__((ext_vector_type(4)));
            const f4v x = {__uint_as_float(v[h]), __uint_as_float(v[(h + 1) % G]), __uint_as_float(v[(h + 2) % G]),
                           __uint_as_float(v[(h + 3) % G])};
            __builtin_nontemporal_store(x, reinterpret_cast<f4v*>(dst + 16 * h));
        }
    } else if (G == 2 && (t_global & 1) == 0) {
        *reinterpret_cast<float2*>(dst) = make_float2(__uint_as_float(v[0]), __uint_as_float(v[1 % G]));
    } else {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int tg = t_global + g;
            a.V[v_index(c, tg, groups)] = __uint_as_float(v[g]);
        }
    }
}

template <int DEPTH, int G>
__device__ __forceinline__ void walk_group(const uint8_t* __restrict__ L, const TreeArgs& a, int t, int t_global,
                                           uint32_t fb, int64_t c, bool active) {
    uint32_t v[G];
    walk_vals<DEPTH, G>(L, a, t, fb, v);
    if (active) store_vals<G>(a, t_global, c, v);
}

// r (< 2H) remaining trees from local tree t, in groups of H, H/2, ..., 1.
template <int DEPTH, int H>
__device__ __forceinline__ void walk_tail(const uint8_t* __restrict__ L, const TreeArgs& a, int t, int t_global, int r,
                                          uint32_t fb, int64_t c, bool active) {
    if (r >= H) {
        walk_group<DEPTH, H>(L, a, t, t_global, fb, c, active);
        t += H;
        t_global += H;
        r -= H;
    }
    if constexpr (H > 1) walk_tail<DEPTH, H / 2>(L, a, t, t_global, r, fb, c, active);
}

// Workgroup b walks trees [g*tpw, g*tpw + tpw) for chain blocks (64 chains
// each) [cs*slice_blocks, (cs+1)*slice_blocks), with g = b / slices and
// cs = b % slices.  Wave w starts with block w of the slice and then takes
// the next unclaimed block from a counter in LDS, so waves that share a
// SIMD with fewer others take more blocks.
// QT: the tile's quads when known at compile time (the whole-feature tiles),
// else 0 (a.q).  ONE: the plan puts one group of G trees on each workgroup.
template <int DEPTH, int QT, bool ONE>
__global__ __launch_bounds__(TREE_WAVES_MAX * 64) void k_trees(TreeArgs a) {
    constexpr int G = 8;
    const int tq = QT ? QT : a.q;
    __shared__ uint32_t lds[MAX_LDS_BYTES / 4];
    const uint8_t* L = reinterpret_cast<const uint8_t*>(lds);
    const int tid = threadIdx.x;
    const int grp = blockIdx.x / a.slices, cs = blockIdx.x - grp * a.slices;
    const int t0 = grp * a.tpw;
    const int nt = (a.n_trees - t0 < a.tpw) ? (a.n_trees - t0) : a.tpw;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int nw = (int)(blockDim.x >> 6);
    uint32_t* counter = lds + a.counter / 4;
    const int64_t n = a.n;
    const int64_t blocks = (n + 63) >> 6;
    const int64_t b_end0 = (int64_t)(cs + 1) * a.slice_blocks;
    const int64_t b_end = b_end0 < blocks ? b_end0 : blocks;
    uint32_t* tile = lds + wave * (a.slot / 4);
    const uint32_t fb = (uint32_t)wave * a.slot + (uint32_t)lane * 4u;
    // tile fill straight from global memory into LDS: instruction k moves
    // quads 4k..4k+3, lane i the 16 bytes of chains 4(i & 15) .. +3 of quad
    // 4k + i/16, which land on tile dwords 256k + 4i .. +3 = quad * 64 + chain
    // (in a last, partial group the lanes past the last quad stay idle)
    const uint32_t* fsrc = a.Fg + (int64_t)(lane >> 4) * a.fg_stride + 4 * (lane & 15);
    const int full = tq >> 2;
    const bool part = (lane >> 4) < (tq & 3);
    auto fill = [&](int64_t blk) {
        const uint32_t* src = fsrc + blk * 64;
        int k = 0;
        for (; k < full; ++k) __builtin_amdgcn_global_load_lds(src + (int64_t)(4 * k) * a.fg_stride, tile + 256 * k, 16, 0, 0);
        if (part) __builtin_amdgcn_global_load_lds(src + (int64_t)(4 * k) * a.fg_stride, tile + 256 * k, 16, 0, 0);
    };
    const int64_t b_first = (int64_t)cs * a.slice_blocks;
    const int64_t nblk = b_end - b_first;
    int64_t r = wave;
    // the first block's tile is in flight while the trees are copied
    if (r < nblk) fill(b_first + r);
    // Trees, already relocated for this LDS plan (a.words32 holds per tree
    // its node block, whose node words carry the LDS addresses of their
    // children, then its leaf block), go block by block straight into LDS:
    // unit u is piece p (PIECE bytes) of block k (node, leaf) of local tree t.
    {
        constexpr uint32_t BB = 4u << DEPTH;                // bytes per block
        constexpr uint32_t SZ = BB >= 16u ? 16u : 4u;       // bytes per lane
        constexpr uint32_t PIECE = 64u * SZ;
        constexpr int PPB = (int)((BB + PIECE - 1u) / PIECE);
        const int units = nt * 2 * PPB;
        for (int u = wave; u < units; u += nw) {
            const int t = u / (2 * PPB), r = u - t * (2 * PPB), k = r / PPB, p = r - k * PPB;
            const uint32_t o = a.toff[t];
            const uint32_t dw = (k ? (o >> 16) : (o & 0xffffu)) + (uint32_t)p * (PIECE / 4u);
            const uint32_t* s = a.words32 + ((size_t)(t0 + t) * 2 + (size_t)k) * (BB / 4u) +
                                (size_t)p * (PIECE / 4u) + (size_t)lane * (SZ / 4u);
            // lanes past the end of a block smaller than one piece stay idle
            if ((uint32_t)lane * SZ < BB - (uint32_t)p * PIECE) {
                if constexpr (SZ == 16u)
                    __builtin_amdgcn_global_load_lds(s, lds + dw, 16, 0, 0);
                else
                    __builtin_amdgcn_global_load_lds(s, lds + dw, 4, 0, 0);
            }
        }
    }
    if (tid == 0) *counter = (uint32_t)nw;
    // every wave's copies and its first tile have landed before any wave reads
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    // the roots of the first eight trees and their children's slots: the
    // same for every chain, read once
    constexpr bool ROOTS = DEPTH >= 2;
    uint32_t rnode[G], rlo[G], rhi[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        rnode[g] = rlo[g] = rhi[g] = 0u;
        if (ROOTS && g < nt) {
            rnode[g] = *reinterpret_cast<const uint32_t*>(L + (a.toff[g] & 0xffffu) * 4u);
            const uint64_t pr = *reinterpret_cast<const uint64_t*>(L + (rnode[g] >> 14));
            rlo[g] = (uint32_t)pr;
            rhi[g] = (uint32_t)(pr >> 32);
        }
    }
    auto claim_next = [&]() -> uint32_t {
        uint32_t r = 0;
        if (lane == 0) r = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        return r;
    };
    // r: the block walked now.  At the start of each block the wave claims
    // the one it walks next; the claim's answer arrives during the walk, so
    // it is never waited for, and no wave holds a block it has not started
    // while others run out of work.
    bool first = true;
    // When a workgroup's trees are one group of G (tree index a multiple of
    // four, so a lane's values go out as two 16-byte stores), a block's leaf
    // values are stored after the next block's fill is issued: the wait for
    // the fill (memory operations complete in the order they were issued)
    // then leaves those two stores in flight.  Every block has an active
    // lane 0, so both stores are always issued.
    const bool defer = ONE && ROOTS && nt == G && (t0 & 3) == 0;
    uint32_t pv[G];
    int64_t pc = 0;
    bool pact = false, pend = false;
    while (r < nblk) {
        // every earlier read of this wave's tile has returned before the
        // tile is overwritten (s_waitcnt lgkmcnt(0))
        if (!first) __builtin_amdgcn_s_waitcnt(0xc07f);
        const uint32_t claim = claim_next();
        const int64_t b = b_first + r;
        if (!first) {
            fill(b);
            if (pend) {
                if (pact) store_vals<G>(a, t0, pc, pv);
                __builtin_amdgcn_s_waitcnt(0x0002);     // vmcnt(2) expcnt(0) lgkmcnt(0)
                pend = false;
            } else {
                __builtin_amdgcn_s_waitcnt(0);
            }
        }
        first = false;
        const int64_t c = b * 64 + lane;
        const bool active = c < n;
        int t = 0;
        if (ROOTS && nt >= G) {
            uint32_t nbr[G], v[G];
#pragma unroll
            for (int g = 0; g < G; ++g) nbr[g] = 0u;
            walk8_roll<(ROOTS ? DEPTH : 2), true>(L, nbr, fb, a.mask, rnode, rlo, rhi, v);
            if (defer) {
#pragma unroll
                for (int g = 0; g < G; ++g) pv[g] = v[g];
                pc = c;
                pact = active;
                pend = true;
            } else if (active) {
                store_vals<G>(a, t0, c, v);
            }
            t = G;
        }
        for (; t + G <= nt; t += G) walk_group<DEPTH, G>(L, a, t, t0 + t, fb, c, active);
        walk_tail<DEPTH, G / 2>(L, a, t, t0 + t, nt - t, fb, c, active);
        r = (int64_t)__builtin_amdgcn_readfirstlane(claim);
    }
    if (pend && pact) store_vals<G>(a, t0, pc, pv);
}

// The pointer form relocated for one LDS plan and tile layout.  Word j of a
// tree holds heap node j (the root, node 1, is word 0; word 1 is unused;
// leaves are words 2^DEPTH and up), so node j's parent is node j / 2.
//  - Settling: when a node's feature is constant over the space (fmap
//    entry 0x100 | value), the child it reaches is known, and both of its
//    children become that child (the slot's other word takes a copy of it),
//    so the walk reaches the same leaf whatever the tile holds there.
//  - Every node word gets its feature's tile position (position 0 for a
//    settled node, whose byte is read but decides nothing) and, in its high
//    half, the LDS word address of the block its children's slot lies in
//    (local tree t % tpw; the leaf block for slots p >= NB / 2, whose nodes
//    are on the last internal level, and for the root when DEPTH is 1).
// fmap null: identity tile layout, nothing settled.  Runs once per
// annealing run, so that the tree kernel copies its trees into LDS
// unchanged.
__global__ void k_reloc(const uint32_t* __restrict__ src, uint32_t* __restrict__ dst, int64_t words, int depth,
                        const uint16_t* __restrict__ fmap, TreeArgs a) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= words) return;
    const uint32_t nb = 1u << (depth - 1);
    const int64_t t = i >> (depth + 1);
    const uint32_t j = (uint32_t)(i & ((2 << depth) - 1));
    const uint32_t* tw = src + (t << (depth + 1));
    auto feature_of = [](uint32_t c) { return (c & 3u) | ((c >> 8) << 2); };   // compact node c
    uint32_t js = j;
    if (fmap && j >= 2u) {
        const uint32_t p = j >> 1;
        const uint32_t pc = tw[p == 1u ? 0u : p] & 0xffffu;
        const uint32_t m = fmap[feature_of(pc)];
        if (m & 0x100u) js = (j & ~1u) | ((m & 0xffu) >= ((pc >> 2) & 0x3fu) ? 1u : 0u);
    }
    uint32_t v = tw[js];
    if (j < 2u * nb) {
        if (fmap) {
            const uint32_t c = v & 0xffffu;
            const uint32_t m = fmap[feature_of(c)];
            const uint32_t pos = (m & 0x100u) ? 0u : m;
            v = (v & 0xffff00fcu) | (pos & 3u) | ((pos >> 2) << 8);
        }
        const uint32_t o = a.toff[t % a.tpw];
        v += ((j >> 1) >= nb / 2u ? (o >> 16) : (o & 0xffffu)) << 16;
    }
    dst[i] = v;
}

// LDS plan of a tree workgroup: nw feature tiles of Q quads, one per slot,
// the block counter (16 bytes: at the end of the LDS, or with in_slot in the
// first slot's spare bytes), and the node and leaf blocks of tpw trees placed
// first-fit (largest first) in the space left free.  Returns false when they
// do not fit.
bool plan_trees(int depth, int Q, uint32_t slot, int nw, int tpw, bool in_slot, uint32_t (&toff)[TREES_MAX],
                uint32_t& counter) {
    const uint32_t tile = (uint32_t)Q * 256u;
    if (in_slot && (nw < 2 || slot - tile < 16u)) return false;
    counter = in_slot ? slot - 16u : (uint32_t)MAX_LDS_BYTES - 16u;
    const uint32_t end = in_slot ? (uint32_t)MAX_LDS_BYTES : (uint32_t)MAX_LDS_BYTES - 16u;
    struct Gap { uint32_t lo, hi; };
    Gap gaps[TREE_WAVES_MAX];
    int ng = 0;
    for (int w = 0; w < nw; ++w) {
        const uint32_t lo = (uint32_t)w * slot + tile;
        const uint32_t hi = (w + 1 < nw) ? (w == 0 && in_slot ? counter : (uint32_t)(w + 1) * slot) : end;
        if (lo > end) return false;
        gaps[ng++] = Gap{lo, hi};
    }
    // node and leaf blocks: 2^(depth-1) slots of 8 bytes each
    const uint32_t nbytes = 4u << depth, lbytes = 4u << depth;
    uint32_t noff[TREES_MAX], loff[TREES_MAX];
    auto place = [&](uint32_t bytes, uint32_t& off) {
        for (int i = 0; i < ng; ++i) {
            if (gaps[i].hi - gaps[i].lo >= bytes) {
                off = gaps[i].lo;
                gaps[i].lo += bytes;
                return true;
            }
        }
        return false;
    };
    for (int t = 0; t < tpw; ++t)
        if (!place(lbytes, loff[t])) return false;
    for (int t = 0; t < tpw; ++t)
        if (!place(nbytes, noff[t])) return false;
    // every block clear of the tiles and the counter
    auto clear = [&](uint32_t off, uint32_t bytes) {
        if (off + bytes > (uint32_t)MAX_LDS_BYTES) return false;
        if (off < counter + 16u && counter < off + bytes) return false;
        for (int w = 0; w < nw; ++w)
            if (off < (uint32_t)w * slot + tile && (uint32_t)w * slot < off + bytes) return false;
        return true;
    };
    for (int t = 0; t < tpw; ++t)
        if (!clear(loff[t], lbytes) || !clear(noff[t], nbytes)) return false;
    for (int t = 0; t < tpw; ++t) toff[t] = (noff[t] / 4u) | ((loff[t] / 4u) << 16);
    return true;
}

template <int DEPTH, int QT, bool ONE>
hipError_t launch_trees_t(const TreeArgs& a, int nw, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
    const int grid = (a.n_trees + a.tpw - 1) / a.tpw * a.slices;
    static bool checked = false;
    if (!checked) {
        // the walk's asm takes offsets into the kernel's LDS array as LDS
        // addresses: the array must be the kernel's only LDS object
        hipFuncAttributes fa;
        hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void*>(&k_trees<DEPTH, QT, ONE>));
        if (e != hipSuccess) return e;
        if (fa.sharedSizeBytes != MAX_LDS_BYTES) return hipErrorInvalidKernelFile;
        checked = true;
    }
    if (start)
        hipExtLaunchKernelGGL((k_trees<DEPTH, QT, ONE>), dim3(grid), dim3(nw * 64), 0, stream, start, stop, 0, a);
    else
        hipLaunchKernelGGL((k_trees<DEPTH, QT, ONE>), dim3(grid), dim3(nw * 64), 0, stream, a);
    return hipGetLastError();
}

template <int QT, bool ONE>
hipError_t launch_trees_o(const TreeArgs& a, int depth, int nw, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop) {
    switch (depth) {
        case 1: return launch_trees_t<1, QT, ONE>(a, nw, stream, start, stop);
        case 2: return launch_trees_t<2, QT, ONE>(a, nw, stream, start, stop);
        case 3: return launch_trees_t<3, QT, ONE>(a, nw, stream, start, stop);
        case 4: return launch_trees_t<4, QT, ONE>(a, nw, stream, start, stop);
        case 5: return launch_trees_t<5, QT, ONE>(a, nw, stream, start, stop);
        case 6: return launch_trees_t<6, QT, ONE>(a, nw, stream, start, stop);
        case 7: return launch_trees_t<7, QT, ONE>(a, nw, stream, start, stop);
        case 8: return launch_trees_t<8, QT, ONE>(a, nw, stream, start, stop);
        case 9: return launch_trees_t<9, QT, ONE>(a, nw, stream, start, stop);
        case 10: return launch_trees_t<10, QT, ONE>(a, nw, stream, start, stop);
        case 11: return launch_trees_t<11, QT, ONE>(a, nw, stream, start, stop);
        case 12: return launch_trees_t<12, QT, ONE>(a, nw, stream, start, stop);
        default: return hipErrorInvalidValue;
    }
}

// Workgroups of one group of trees (eight) keep a block's leaf values until
// the next block's fill is issued.
template <int QT>
hipError_t launch_trees_q(const TreeArgs& a, int depth, int nw, hipStream_t stream, hipEvent_t start,
                          hipEvent_t stop) {
    return a.tpw == 8 ? launch_trees_o<QT, true>(a, depth, nw, stream, start, stop)
                      : launch_trees_o<QT, false>(a, depth, nw, stream, start, stop);
}

// Whole-feature tiles (GEMM and conv2d loop-context rows, relation rows)
// have their quad count compiled in; compact tiles take it at run time.
hipError_t launch_trees(const TreeArgs& a, int depth, int nw, hipStream_t stream, hipEvent_t start, hipEvent_t stop) {
    switch (a.q) {
        case 28: return launch_trees_q<28>(a, depth, nw, stream, start, stop);
        case 44: return launch_trees_q<44>(a, depth, nw, stream, start, stop);
        case REL_Q: return launch_trees_q<REL_Q>(a, depth, nw, stream, start, stop);
        default: return launch_trees_q<0>(a, depth, nw, stream, start, stop);
    }
}

// Tile slot of Q quads: the smallest power of two holding Q * 256 bytes.
uint32_t slot_bytes(int Q) {
    uint32_t s = 256u;
    while (s < (uint32_t)Q * 256u) s <<= 1;
    return s;
}

// Launch plan of the tree kernel for an ensemble walked over Q-quad tiles of
// n chains: tree groups of tpw trees times chain slices, the layout scoring
// the walks in flight per compute unit (waves times trees walked together)
// times the share of compute units its grid fills.  Fills ta's plan fields
// and nw; false when nothing fits.
bool plan_tree_launch(int n_trees, int depth, int Q, int64_t n, int n_cu, TreeArgs& ta, int& nw) {
    const uint32_t slot = slot_bytes(Q);
    const int64_t blocks = (n + 63) / 64;
    double best_score = -1.0;
    nw = 0;
    for (int tpw = TREES_MAX; tpw >= 1; tpw /= 2) {
        const int tg = (n_trees + tpw - 1) / tpw;
        int64_t slices = n_cu / tg;
        if (slices < 1) slices = 1;
        if (slices > blocks) slices = blocks;
        const int64_t sb = (blocks + slices - 1) / slices;
        slices = (blocks + sb - 1) / sb;
        const int cap = sb < TREE_WAVES_MAX ? (int)sb : TREE_WAVES_MAX;
        uint32_t toff[TREES_MAX], counter = 0;
        for (int w = cap; w >= 1; --w) {
            // the counter at the end of the LDS, or in a tile slot's spare
            // bytes when only that leaves room
            if (!plan_trees(depth, Q, slot, w, tpw, false, toff, counter) &&
                !plan_trees(depth, Q, slot, w, tpw, true, toff, counter))
                continue;
            const double grid = (double)tg * (double)slices;
            const double score = (double)w * (tpw < 8 ? tpw : 8) * (grid < n_cu ? grid / n_cu : 1.0);
            if (score > best_score) {
                best_score = score;
                nw = w;
                ta.tpw = tpw;
                ta.slices = (int)slices;
                ta.slice_blocks = (int)sb;
                ta.counter = counter;
                for (int i = 0; i < TREES_MAX; ++i) ta.toff[i] = toff[i];
            }
            break;
        }
    }
    if (nw == 0) return false;
    ta.q = Q;
    ta.slot = slot;
    ta.mask = ((slot - 1u) & ~0xffu) | 3u;
    return true;
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

// Start and stop events for the next launch of one kind, or nulls when the
// chains are not being profiled.
hipError_t next_events(at_chains_s& ch, int kind, hipEvent_t& start, hipEvent_t& stop) {
    start = stop = nullptr;
    if (!ch.profiling) return hipSuccess;
    std::vector<hipEvent_t>& pool = ch.events[kind];
    size_t& used = ch.events_used[kind];
    while (pool.size() < used + 2) {
        hipEvent_t e;
        hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return err;
        pool.push_back(e);
    }
    start = pool[used];
    stop = pool[used + 1];
    used += 2;
    return hipSuccess;
}

// One ensemble's tree kernel for a run: its plan, its pointer form
// relocated for that plan, and the tile and leaf-value buffers it uses.
struct TreeLaunch {
    TreeArgs ta{};
    int nw = 0;
    int depth = 0;
};

// Q: quads per chain in a tile; fmap: the space's tile layout (null for
// the relation features, which are tiled whole).
static hipError_t prepare_trees(const EnsembleDesc& e, int Q, const uint16_t* fmap, int64_t n, int n_cu,
                                DeviceBuf& relocated, const uint32_t* Fg, int64_t fg_stride, float* V,
                                hipStream_t stream, TreeLaunch& tl) {
    tl.depth = e.depth;
    TreeArgs& ta = tl.ta;
    ta.words32 = e.words32;
    ta.n_trees = e.n_trees;
    ta.Fg = Fg;
    ta.fg_stride = fg_stride;
    ta.n = n;
    ta.V = V;
    if (!plan_tree_launch(e.n_trees, e.depth, Q, n, n_cu, ta, tl.nw)) return hipErrorInvalidConfiguration;
    const int64_t words = (int64_t)e.n_trees << (e.depth + 1);
    hipError_t err = ensure(relocated, (size_t)words * 4);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_reloc, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, stream, e.words32,
                       static_cast<uint32_t*>(relocated.p), words, e.depth, fmap, ta);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    ta.words32 = static_cast<const uint32_t*>(relocated.p);
    return hipSuccess;
}

hipError_t launch_sa_tp(const at_space_s& sp, const EnsembleDesc& e, const EnsembleDesc* eg, at_chains_s& ch,
                        int steps, bool init, const float* thr, at_entry* best, at_entry* trace, hipStream_t stream) {
    const int64_t n = ch.n_chains;
    if (n == 0) return hipSuccess;
    const int Q = (sp.descs[0].n_features + 3) / 4;
    const int groups = (e.n_trees + 3) / 4;
    const int64_t n16 = (n + 15) / 16 * 16;
    hipError_t err;
    if ((err = ensure(ch.d_cand, (size_t)n * MAX_KNOBS * 2)) != hipSuccess) return err;
    if ((err = ensure(ch.d_meta, (size_t)n * sizeof(ChainMeta))) != hipSuccess) return err;
    const int64_t fg_stride = (n + 63) / 64 * 64;
    if ((err = ensure(ch.d_fg, (size_t)Q * fg_stride * 4)) != hipSuccess) return err;
    if ((err = ensure(ch.d_v, (size_t)groups * n16 * 16)) != hipSuccess) return err;
    if (eg) {
        if ((err = ensure(ch.d_fr, (size_t)REL_Q * fg_stride * 4)) != hipSuccess) return err;
        if ((err = ensure(ch.d_vg, (size_t)((eg->n_trees + 3) / 4) * n16 * 16)) != hipSuccess) return err;
    }

    ChainArgs ca{};
    ca.descs = static_cast<const SpaceDesc*>(sp.d_descs.p);
    ca.offsets = static_cast<const int64_t*>(sp.d_offsets.p);
    ca.n_spaces = sp.n_spaces;
    ca.factors = static_cast<const uint64_t*>(sp.d_factors.p);
    ca.stage = static_cast<const uint8_t*>(sp.d_stage.p);
    ca.stage_stride = sp.stage_stride;
    ca.stage_single = sp.stage_single;
    ca.wg_space = static_cast<const int32_t*>(sp.d_wg_space.p);
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
    ca.fg_stride = fg_stride;
    ca.steps = steps;
    ca.thr = thr;
    ca.trace = trace;
    ca.fsrc = static_cast<const uint8_t*>(sp.d_fsrc.p);
    ca.fq = sp.tile_q;
    ca.fident = sp.tile_q == Q ? 1 : 0;
    if (eg) {
        ca.Vg = static_cast<const float*>(ch.d_vg.p);
        ca.Tg = eg->n_trees;
        ca.Fr = static_cast<uint32_t*>(ch.d_fr.p);
    }

    int n_cu = 256;
    (void)hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, ch.device);
    // the local (or only) model over the loop features, then the global model
    // over the relation features
    TreeLaunch tl, tg;
    if ((err = prepare_trees(e, sp.tile_q, static_cast<const uint16_t*>(sp.d_fmap.p), n, n_cu, ch.d_tw, ca.Fg,
                             fg_stride, static_cast<float*>(ch.d_v.p), stream, tl)) != hipSuccess)
        return err;
    if (eg && (err = prepare_trees(*eg, REL_Q, nullptr, n, n_cu, ch.d_twg, ca.Fr, fg_stride,
                                   static_cast<float*>(ch.d_vg.p), stream, tg)) != hipSuccess)
        return err;

    const unsigned chain_grid = (unsigned)((n + CPW - 1) / CPW);
    const size_t chain_lds = ring_bytes(eg != nullptr) + (size_t)CPW * ch.topk * sizeof(at_entry);
    {
        const TreeArgs& ta = tl.ta;
        const int64_t tree_grid = (int64_t)(e.n_trees + ta.tpw - 1) / ta.tpw * ta.slices;
        const int64_t plan[8] = {ta.tpw, tl.nw, tree_grid, ta.slices, ta.slice_blocks, (int64_t)chain_grid,
                                 (int64_t)ta.q, (int64_t)groups * n16 * 16};
        for (int i = 0; i < 8; ++i) ch.last_plan[i] = plan[i];
    }
    static bool chain_configured = false;
    if (!chain_configured) {
        for (const void* f : {reinterpret_cast<const void*>(&k_chain<AT_TMPL_GEMM, 256>),
                              reinterpret_cast<const void*>(&k_chain<AT_TMPL_CONV2D_NCHW, 256>),
                              reinterpret_cast<const void*>(&k_chain<AT_TMPL_GEMM, 512>),
                              reinterpret_cast<const void*>(&k_chain<AT_TMPL_CONV2D_NCHW, 512>)}) {
            if ((err = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)(ring_bytes(true) + (size_t)CPW * KMAX * sizeof(at_entry)))) != hipSuccess)
                return err;
        }
        chain_configured = true;
    }
    ch.events_used[0] = ch.events_used[1] = 0;
    // While wave 0 folds, the other waves build both next candidates of 16
    // chains (2 x 16 x L loop-feature tasks).  With a short fold (under 1500
    // trees in all) that building is the longer of the two and eight waves
    // take it (twelve conv2d workloads, 1000 trees: 14.2 -> 13.3 ms a run);
    // with a long fold four waves leave the folding wave more of its SIMD
    // (C12, 2000 trees: 56.6 against 57.1 ms).
    const bool wide = e.n_trees + (eg ? eg->n_trees : 0) < 1500;
    auto chain_kernel = [&](const ChainArgs& x) -> hipError_t {
        const size_t lds = x.fin == FIN_NONE ? 0 : chain_lds;
        hipEvent_t start, stop;
        const hipError_t ev = next_events(ch, 1, start, stop);
        if (ev != hipSuccess) return ev;
        auto kern = sp.tmpl == AT_TMPL_GEMM ? (wide ? k_chain<AT_TMPL_GEMM, 512> : k_chain<AT_TMPL_GEMM, 256>)
                                            : (wide ? k_chain<AT_TMPL_CONV2D_NCHW, 512> : k_chain<AT_TMPL_CONV2D_NCHW, 256>);
        const int wg = wide ? 512 : 256;
        if (start)
            hipExtLaunchKernelGGL(kern, dim3(chain_grid), dim3(wg), lds, stream, start, stop, 0, x);
        else
            hipLaunchKernelGGL(kern, dim3(chain_grid), dim3(wg), lds, stream, x);
        return hipGetLastError();
    };
    auto trees_kernel = [&]() -> hipError_t {
        for (const TreeLaunch* t : {eg ? &tg : nullptr, &tl}) {
            if (!t) continue;
            hipEvent_t start, stop;
            hipError_t ev = next_events(ch, 0, start, stop);
            if (ev != hipSuccess) return ev;
            if ((ev = launch_trees(t->ta, t->depth, t->nw, stream, start, stop)) != hipSuccess) return ev;
        }
        return hipSuccess;
    };

    int pending = FIN_NONE;
    if (init) {
        ChainArgs x = ca;
        x.fin = FIN_NONE;
        x.draw = DRAW_INIT;
        if ((err = chain_kernel(x)) != hipSuccess) return err;
        if ((err = trees_kernel()) != hipSuccess) return err;
        pending = FIN_INIT;
    }
    for (int s = 0; s < steps; ++s) {
        ChainArgs x = ca;
        x.fin = pending;
        x.fin_step = s - 1;
        x.draw = DRAW_PROPOSE;
        x.draw_step = (uint32_t)(ch.step_abs + (uint64_t)s);
        if (!eg && !wide) {
            // a long fold leaves the building waves time to spare: they bring
            // the next tree launch's trees into the L2 (with a short fold the
            // building is the longer side and this would lengthen the step)
            x.pf_trees = reinterpret_cast<const uint8_t*>(tl.ta.words32);
            x.pf_tree_bytes = 8 << e.depth;
            x.pf_tpw = tl.ta.tpw;
            x.pf_ntrees = e.n_trees;
        }
        if ((err = chain_kernel(x)) != hipSuccess) return err;
        if ((err = trees_kernel()) != hipSuccess) return err;
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
