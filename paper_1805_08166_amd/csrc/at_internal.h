// Internal declarations of the autotensor library (not part of the C ABI).
//
// Device-side descriptions of schedule spaces, packed tree ensembles and
// annealing chains, plus the Philox-4x32-10 block function shared by the
// host threshold helper and the kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/autotensor.h"

namespace at {

// Knobs of a space: splits (one per axis), auto_unroll_max_step,
// unroll_explicit, and for the annotated templates vectorize and vthread
// (conv2d: 6 + 2 + 2).  Chains keep their knob vectors as 12 u16 (24 bytes).
constexpr int MAX_KNOBS = 12;
constexpr int MAX_AXES = 6;
constexpr int N_BUFFERS = 3;
// Lanes of one feature tile in LDS.  A tile holds the u8 features of 256
// rows "quad-major": byte (f & 3) of dword (f >> 2) * 256 + lane, so every
// lane of a wave reads its own bank whatever feature it asks for.
constexpr int TILE_LANES = 256;
constexpr int MAX_TILE_QUADS = 64;   // up to 256 features
// Context relation features per configuration (Section 4): 2 pairs x 3
// buffers x 32 thresholds.
constexpr int RELATION_FEATURES = 192;
// Packed ensembles are zero-padded to a multiple of this many words.
constexpr size_t ENSEMBLE_PAD_WORDS = 8192;

// Schedule space as the kernels see it.  Split knobs come first (one per
// axis, axis a is knob a), then auto_unroll_max_step, then unroll_explicit.
struct SpaceDesc {
    int32_t tmpl;
    int32_t n_knobs;
    int32_t n_axes;
    int32_t n_features;
    int32_t n_mut;                       // knobs with at least two values
    int32_t mut[MAX_KNOBS];              // their indices, ascending
    uint32_t knob_size[MAX_KNOBS];
    uint64_t n_configs;
    uint64_t radix[MAX_KNOBS];           // product of the sizes of later knobs
    int32_t split_off[MAX_AXES];         // split choices of axis a start at
                                         // factors[split_off[a]] (u64 each)
    int32_t coef[N_BUFFERS][MAX_AXES];   // weight of axis a in buffer b's flat index
    int32_t stride;                      // conv stride S (1 for GEMM)
    int32_t ann_knobs;                   // 1: knobs n_axes + 2, n_axes + 3 are vectorize and vthread
};

// LDS image of one space for the annealing chain kernel: the descriptor
// with its split offsets rebased to 0 in the first STAGE_DESC_BYTES, then
// the space's split factors (u64), at most STAGE_FAC_MAX of them.  Images
// of a space set lie STAGE_ALIGN-multiple strides apart; the kernel copies
// a whole stride with 16-byte direct-to-LDS moves of whole waves.
constexpr int STAGE_DESC_BYTES = (int)((sizeof(SpaceDesc) + 15) / 16 * 16);
constexpr int STAGE_FAC_MAX = 1024;
constexpr int STAGE_ALIGN = 1024;
constexpr int STAGE_MAX_BYTES = (STAGE_DESC_BYTES + STAGE_FAC_MAX * 8 + STAGE_ALIGN - 1) / STAGE_ALIGN * STAGE_ALIGN;
constexpr int STAGE_CHAINS = 16;         // chains per chain-kernel workgroup

// Packed ensemble.  Tree t occupies words [t*W, (t+1)*W) with W = 2^(d+1):
// word m (1 <= m < 2^d) is internal node m (1-based heap order: children 2m
// and 2m+1) holding (thr << 16) | tile byte offset of its feature; words
// 2^d .. 2^(d+1)-1 hold the leaf values (float bits); word 0 is unused.
//
// The annealing path uses a second, compact form (words16): its features
// are loop-context bitlens, never above 31, so a split on x < thr decides
// the same with thr clamped to 32.  Tree t occupies words16 [t*W16,
// (t+1)*W16) with W16 = 3 * 2^(d-1): a node block of 2^(d-1) words (word 0
// holds the root in its low half, word p >= 1 holds internal nodes 2p and
// 2p+1 as the low and high halves) followed by the 2^d leaf values.  A
// 16-bit node is (f & 3) | min(thr, 32) << 2 | (f >> 2) << 8.
struct EnsembleDesc {
    int32_t n_trees;
    int32_t depth;
    int32_t n_features;
    int32_t words_per_tree;
    const uint32_t* words;
    const uint32_t* words16;
    // Local forms for the chain-local annealing path: the compact form's
    // trees re-laid at an odd word stride (the smallest >= the tree's words
    // that is 1 mod 32), whole trees (local_full) or node blocks only
    // (local_nodes); zero padded, plus 16 bytes of slack at the end.
    const uint32_t* local_full;
    const uint32_t* local_nodes;
    // Split form for walks whose top levels stay in LDS: local_top holds the
    // first 2^(d-2) words of each compact node block (levels 0 .. d-2) at an
    // odd word stride; tail holds per tree and last-level node m (2^(d-1)
    // of them) a 16-byte record {node m's 16-bit node, its left leaf, its
    // right leaf, 0}.  Depth 2 and above.
    const uint32_t* local_top;
    const uint4* tail;
    // Pointer form for the tree-partitioned annealing path.  Tree t occupies
    // words32 [t*W32, (t+1)*W32) with W32 = 2^(d+1): a node block of 2^(d-1)
    // 8-byte slots (slot 0 holds the root in its low word, slot p >= 1 holds
    // internal nodes 2p and 2p+1), then a leaf block of 2^(d-1) slots (slot j
    // holds leaves 2j and 2j+1).  A 32-bit node is its 16-bit compact node in
    // the low half and, in the high half, the word offset of its children's
    // slot: 2m in the node block for node m < 2^(d-1), 2(m - 2^(d-1)) in the
    // leaf block otherwise.  A kernel that copies the blocks to LDS adds the
    // word address of the target block to the high half, which then holds
    // the LDS address of the children divided by 4.
    const uint32_t* words32;
};

// Largest threshold the compact form keeps; annealing features never exceed
// SA_FEATURE_MAX.
constexpr uint32_t SA_FEATURE_MAX = 31;
constexpr uint32_t SA_THR_CLAMP = SA_FEATURE_MAX + 1;
__host__ __device__ inline uint32_t node16(uint32_t f, uint32_t thr) {
    const uint32_t t = thr < SA_THR_CLAMP ? thr : SA_THR_CLAMP;
    return (f & 3u) | (t << 2) | ((f >> 2) << 8);
}

// Per-chain best-list bookkeeping kept between kernels: number of valid
// entries and the last (k-th) entry.
struct ChainMeta {
    uint32_t count;
    float kth_score;
    uint64_t kth_cfg;
};

// Tile byte offset of feature f: quad (f >> 2), byte (f & 3).
__host__ __device__ inline uint32_t tile_offset(int f) {
    return (uint32_t)((f >> 2) * TILE_LANES * 4 + (f & 3));
}

// --------------------------------------------------------------------------
// Philox-4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 32x32 -> 64-bit products with multipliers 0xD2511F53 / 0xCD9E8D57 and a
// Weyl key schedule with increments 0x9E3779B9 / 0xBB67AE85.
// --------------------------------------------------------------------------
struct U4 { uint32_t x, y, z, w; };

__host__ __device__ inline uint32_t mul_hi32(uint32_t a, uint32_t b) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __umulhi(a, b);
#else
    return (uint32_t)(((uint64_t)a * b) >> 32);
#endif
}

__host__ __device__ inline U4 philox(uint32_t k0, uint32_t k1, U4 c) {
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        uint32_t hi0 = mul_hi32(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
        uint32_t hi1 = mul_hi32(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
        c = U4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return c;
}

// floor(r * n / 2^32): a uniform value in [0, n) from one 32-bit word.
__host__ __device__ inline uint32_t uniform_below(uint32_t r, uint32_t n) { return mul_hi32(r, n); }

// --------------------------------------------------------------------------
// Library handles.
// --------------------------------------------------------------------------
struct DeviceBuf {
    void* p = nullptr;
    size_t bytes = 0;
};

}  // namespace at

struct at_space_s {
    int device = 0;
    int tmpl = 0;                           // template of the loop nest (AT_TMPL_GEMM or AT_TMPL_CONV2D_NCHW)
    int api_tmpl = 0;                       // template id the space was created with (0 .. 3)
    int n_spaces = 1;                       // > 1 for a space set
    std::vector<at::SpaceDesc> descs;       // host copies
    std::vector<int64_t> chain_offsets;     // [n_spaces + 1] (sets only)
    at::DeviceBuf d_descs;                  // SpaceDesc[n_spaces]
    at::DeviceBuf d_factors;                // uint64 split factor tables
    at::DeviceBuf d_offsets;                // int64 [n_spaces + 1]
    at::DeviceBuf d_errors;                 // uint64 out-of-range counter
    // LDS images of the member spaces (stage_stride bytes apart, 0 when no
    // member's image fits), and which image a block of STAGE_CHAINS chains
    // uses: stage_single for a single space, d_wg_space (int32 per block) for
    // a set; -1 when the block spans two spaces or its space's image does not
    // fit
    at::DeviceBuf d_stage;
    int stage_stride = 0;
    int stage_single = -1;
    at::DeviceBuf d_wg_space;
    // per member space: its factor tables as host data (for building sets)
    std::vector<std::vector<uint64_t>> host_factors;
    // Loop-context features constant over the space (set): fconst[f] is the
    // value every configuration gives feature f, 0xff when it varies; empty
    // when the space was too large to scan.
    std::vector<uint8_t> fconst;
    // Feature tiles of the tree-partitioned path: tile_q quads (4 features)
    // per chain.  d_fsrc (uint8 [4 * tile_q]) names the feature at each tile
    // position (0xff: padding); d_fmap (uint16 [256]) gives each feature's
    // tile position, or 0x100 | value for a constant feature, whose tree
    // nodes are settled when the trees are relocated.
    int tile_q = 0;
    at::DeviceBuf d_fsrc;
    at::DeviceBuf d_fmap;
};

struct at_ensemble_s {
    int device = 0;
    at::EnsembleDesc desc{};
    at::DeviceBuf d_words;
    at::DeviceBuf d_words16;
    at::DeviceBuf d_words32;
    at::DeviceBuf d_local_full;
    at::DeviceBuf d_local_nodes;
    at::DeviceBuf d_local_top;
    at::DeviceBuf d_tail;
};

struct at_chains_s {
    int device = 0;
    int64_t chain0 = 0;
    int64_t n_chains = 0;
    int topk = 0;
    uint64_t seed = 0;
    uint64_t step_abs = 0;
    bool initialised = false;
    int n_spaces = 1;
    int tmpl = 0;
    at::DeviceBuf d_knobs;    // uint16 [n_chains][MAX_KNOBS]
    at::DeviceBuf d_score;    // float [n_chains]
    at::DeviceBuf d_top;      // at_entry [n_chains][topk]
    at::DeviceBuf d_descs;    // copy of the space's SpaceDesc[n_spaces]
    at::DeviceBuf d_offsets;  // copy of the space's chain offsets
    // workspace of the tree-partitioned annealing path
    at::DeviceBuf d_cand;     // uint16 [n_chains][MAX_KNOBS] candidates
    at::DeviceBuf d_meta;     // ChainMeta [n_chains]
    at::DeviceBuf d_fg;       // uint32 [Q][n_chains] packed candidate features
    at::DeviceBuf d_v;        // float leaf values, [ceil(T/4)][n_chains][4]
    at::DeviceBuf d_tw;       // uint32 pointer-form trees relocated for the tree kernel's LDS plan
    // Eq. 4 runs (tree-partitioned): the global model's side
    at::DeviceBuf d_fr;       // uint32 [48][n_chains] packed candidate relation features
    at::DeviceBuf d_vg;       // float leaf values of the global model, laid out as d_v
    at::DeviceBuf d_twg;      // the global model's relocated pointer form
    // launch timing (measurement aid): start/stop events attached to every
    // launch of the last run; kind 0 is the tree kernel, 1 the chain kernel
    bool profiling = false;
    std::vector<hipEvent_t> events[2];
    size_t events_used[2] = {0, 0};
    // annealing path: requested (at_sa_path) and taken by the last run
    int path = AT_SA_PATH_AUTO;
    int last_path = AT_SA_PATH_AUTO;
    int64_t last_plan[8] = {0, 0, 0, 0, 0, 0, 0, 0};
};

namespace at {

// Thread-local error message helpers (at_capi.cpp).
at_status fail(at_status st, const std::string& msg);
at_status hip_fail(hipError_t e, const char* what);

// Space construction (at_space.cpp).
at_status build_space(int tmpl, const int64_t* shape, int nshape, SpaceDesc& desc,
                      std::vector<uint64_t>& factors);

// Kernel launchers (at_kernels.hip).
hipError_t launch_extract(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                          hipStream_t stream);
hipError_t launch_extract_onehot(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                 hipStream_t stream);
hipError_t launch_extract_full(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                               hipStream_t stream);
hipError_t launch_relation(const at_space_s& sp, const uint64_t* cfgs, int64_t n, int32_t* feats,
                           hipStream_t stream);
// flags[f] = 1 when loop-context feature f is not the same for every
// configuration of a single space; ref[f] = configuration 0's value.
hipError_t launch_feature_scan(const at_space_s& sp, uint32_t* flags, uint32_t* ref, hipStream_t stream);
// accumulate: add to scores (fp32, the stored value first) instead of storing
hipError_t launch_predict(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores,
                          uint16_t* leaves, bool accumulate, hipStream_t stream);
hipError_t launch_score(const EnsembleDesc& e, const int32_t* feats, int64_t n, float* scores,
                        uint16_t* leaves, bool accumulate, hipStream_t stream);
// eg: the global model of an Eq. 4 run (over the relation features), or null.
hipError_t launch_sa_tp(const at_space_s& sp, const EnsembleDesc& e, const EnsembleDesc* eg, at_chains_s& ch,
                        int steps, bool init, const float* thr, at_entry* best, at_entry* trace, hipStream_t stream);
// Chain-local annealing path (at_sa_local.hip): launch geometry and the
// byte offsets of its dynamic LDS blocks.
struct LocalPlan {
    int cpb = 0;              // chains per workgroup
    int threads = 0;
    int grid = 0;
    int gather = 0;           // leaves read from global memory
    int ts = 0;               // tree stride of the local form used (words)
    int ct = 0;               // trees per chunk
    int n_chunks = 0;         // chunks walked per step
    int resident = 0;         // 1: every tree stays in LDS, loaded once
    int tail = 0;             // 1: tree tops resident in LDS, last level and leaves gathered
    uint32_t ring_bytes = 0;
    int walk_waves = 0;       // waves 1 .. walk_waves walk, later ones load
    uint32_t off_ring = 0, off_lv = 0, off_lists = 0, off_rec = 0, off_frow = 0, off_any = 0, off_desc = 0;
    uint32_t frow_stride = 0; // single-pass modes: bytes between the two feature-row buffers
    int lv_stride = 0;
    size_t lds_bytes = 0;
    double round_bytes = 0.0; // bytes streamed per round by one workgroup
};
int local_tree_stride(int words);
bool plan_local(const at_space_s& sp, const EnsembleDesc& e, const at_chains_s& ch, LocalPlan& pl);
hipError_t launch_sa_local(const at_space_s& sp, const EnsembleDesc& e, at_chains_s& ch, const LocalPlan& pl,
                           int steps, bool init, const float* thr, at_entry* best, at_entry* trace,
                           hipStream_t stream);
// Start and stop events for the next launch of one kind (0: the walk
// kernel, 1: the chain kernel), or nulls when the chains are not profiled.
hipError_t next_events(at_chains_s& ch, int kind, hipEvent_t& start, hipEvent_t& stop);

// Batch selection (at_select.hip).
int select_pool_max();
int select_pick_max();
// scratch: two buffers of select_scratch_max_entries() entries each (the
// device's static scratch), or null for stream-ordered allocations.
hipError_t launch_select(const at_space_s& sp, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                         float alpha, int n_random, uint64_t seed, at_entry* out, hipStream_t stream,
                         at_entry* scratch);
// Entries of each partial-result buffer the reduction needs (0: none).
int64_t select_scratch_entries(int64_t n_cand, int pool);
int64_t select_scratch_max_entries();
// Address of the static selection scratch on `device` (which must be
// current), looked up once per device.
hipError_t select_scratch_ptr(int device, at_entry** out);

hipError_t launch_export(const at_chains_s& ch, uint64_t* cur_cfg, float* cur_score,
                         hipStream_t stream);

}  // namespace at
