/*
 * autotensor.h -- C ABI of the MI355X (gfx950) annealing hot path of
 * "Learning to Optimize Tensor Programs" (Chen et al., NeurIPS 2018).
 *
 * The library explores a schedule template's knob space with many
 * independent simulated-annealing chains whose energy is a gradient-boosted
 * tree cost model over loop-context features (Section 3.3, Algorithm 1;
 * Section 3.1; Appendix A.2).  Every compute call runs hand-written HIP
 * kernels on the GPU; nothing here falls back to the CPU.
 *
 * Conventions shared by every entry point
 *   - Pointers tagged "device" are caller-owned device allocations (HIP
 *     device memory, e.g. PyTorch tensors); "host" pointers are ordinary
 *     host memory.  The caller keeps every buffer alive until the stream work
 *     that uses it has completed.
 *   - Handles (at_space_t, at_ensemble_t, at_chains_t) are library-owned
 *     and released with the matching *_destroy call.  A handle is bound to
 *     the device that was current when it was created.
 *   - Compute calls (at_extract_features, at_gbt_predict, at_sa_run,
 *     at_sa_run_traced, at_chains_export) only enqueue work on the given
 *     stream (0 = the null stream) and return without synchronising.
 *     Create calls are synchronous.
 *   - Every call returns an at_status.  Argument errors are reported before
 *     anything is enqueued.  at_last_error() returns a thread-local message
 *     describing the last non-OK status.
 *   - Layouts are row-major.  Feature rows hold n_features int32 values.
 */
#ifndef AUTOTENSOR_H
#define AUTOTENSOR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct at_space_s* at_space_t;
typedef struct at_ensemble_s* at_ensemble_t;
typedef struct at_chains_s* at_chains_t;
typedef void* at_stream_t; /* a hipStream_t; 0 selects the null stream */

typedef enum {
    AT_OK = 0,
    AT_E_INVALID = -1,     /* bad argument (null pointer, bad size, bad handle) */
    AT_E_UNSUPPORTED = -2, /* shape or size the kernels do not handle */
    AT_E_OOM = -3,         /* device or host allocation failed */
    AT_E_HIP = -4,         /* a HIP runtime call failed */
    AT_E_RANGE = -5,       /* a configuration index outside [0, n_configs) */
    AT_E_MISMATCH = -6     /* space and ensemble feature counts differ, or
                              spaces of one set use different templates */
} at_status;

/* Schedule templates (Section 2).
 *  AT_TMPL_GEMM: C[i,j] = sum_k A[k,i] * B[k,j]; shape {M, N, K}.
 *    Knobs: 4-level split of i, 4-level split of j, 2-level split of k,
 *    auto_unroll_max_step in {0, 512, 1500}, unroll_explicit in {0, 1}.
 *    Nest i1 j1 i2 j2 k1 i3 j3 k2 i4 j4 (i1/j1 -> blockIdx.y/x,
 *    i2/j2 -> threadIdx.y/x): 10 loops, 110 features.
 *  AT_TMPL_CONV2D_NCHW: out[k][oh][ow] = sum_{c,ry,rx}
 *    data_pad[c][oh*S+ry][ow*S+rx] * kernel[k][c][ry][rx];
 *    shape {N, C, H, W, K, KH, KW, pad, stride} with N == 1.
 *    Knobs: 4-level splits of oc, oh, ow; 2-level splits of rc, ry, rx;
 *    auto_unroll_max_step; unroll_explicit.  Nest oc1 oh1 ow1 oc2 oh2 ow2
 *    rc1 r1 oc3 oh3 ow3 rc2 r2 oc4 oh4 ow4 (r_l fuses ry_l, rx_l; first band
 *    -> blockIdx.z/y/x, second -> threadIdx.z/y/x): 16 loops, 176 features.
 *  AT_TMPL_GEMM_VT, AT_TMPL_CONV2D_NCHW_VT: the same templates with two
 *    annotation knobs more (Section 2 lists unrolling and vectorization
 *    among the annotations of its search space), after unroll_explicit:
 *    vectorize in {0, 1} marks the innermost loop (GEMM j4, conv2d ow4)
 *    vectorized, annotation id 10; vthread in {0, 1} binds the third tiling
 *    level of every spatial axis (GEMM i3 j3, conv2d oc3 oh3 ow3) to virtual
 *    threads, annotation id 9.  Either takes the place of the unroll rule on
 *    its loops; nest, buffers and every other feature are unchanged.  7 and
 *    10 knobs, four times as many configurations (index = base index * 4 +
 *    vectorize * 2 + vthread).
 * Ordered splits are enumerated lexicographically (outer level first); a
 * configuration index is the mixed-radix number of the knob values with
 * knob 0 most significant. */
typedef enum {
    AT_TMPL_GEMM = 0,
    AT_TMPL_CONV2D_NCHW = 1,
    AT_TMPL_GEMM_VT = 2,
    AT_TMPL_CONV2D_NCHW_VT = 3
} at_template;

/* One entry of a chain's best list, or of an annealing trace. */
typedef struct {
    uint64_t cfg;   /* configuration index */
    float score;    /* model score (higher is better) */
    uint32_t flag;  /* best list: 1 = valid entry; trace: 1 = move accepted */
} at_entry;

/* Builds the schedule space S_e of an index expression e (Section 2):
 * knob tables, loop nest and buffer index expressions, uploaded once to the
 * current device.  A space of at most 2^28 configurations is also scanned
 * whole on the device (one kernel on the null stream) for the loop-context
 * features that take one value over it: the tree-partitioned annealing
 * path leaves those out of its feature tiles (at_chains_last_plan).
 * shape: host [nshape] int64 (see at_template).
 * Errors: AT_E_INVALID for bad shapes; AT_E_UNSUPPORTED when the nest's
 * iteration count or a buffer size reaches 2^31, or the space holds 2^32 or
 * more configurations.  Synchronous. */
at_status at_space_create(int tmpl, const int64_t* shape, int nshape, at_space_t* out);

/* Metadata of the schedule space S_e (Section 2): the knobs of the
 * configuration s = [s_1 .. s_m] and their value counts, the loop count of
 * the lowered nest and the length of its loop-context feature rows
 * (Appendix A.2), and |S_e|.  knob_sizes: host [at least n_knobs], may be
 * NULL; any other output pointer may be NULL.  AT_E_INVALID for a NULL
 * space.  Host only; nothing is enqueued. */
at_status at_space_info(at_space_t space, int* n_knobs, int32_t* knob_sizes, int* n_loops,
                        int* n_features, uint64_t* n_configs);

/* A set of spaces of one template, for annealing several workloads in one
 * launch (transfer-style search over an invariant representation, Section 4).
 * chain_offsets: host [n + 1] int64, ascending, chain_offsets[0] == 0: space
 * i owns the chains [chain_offsets[i], chain_offsets[i+1]).  The set keeps
 * its own copies of the member spaces' tables; members may be destroyed
 * afterwards.  A loop-context feature counts as constant over the set when
 * every member fixes it at the same value.  AT_E_MISMATCH if the templates
 * differ.  Synchronous. */
at_status at_spaceset_create(const at_space_t* spaces, int n, const int64_t* chain_offsets,
                             at_space_t* out);
void at_space_destroy(at_space_t space);

/* Loop-context features of configurations (Appendix A.2), one row per
 * configuration: per loop (outer to inner) bitlen(length), annotation id,
 * then for each buffer bitlen(touch count), bitlen(reuse ratio),
 * bitlen(stride).  bitlen(x) = 0 for x = 0, else floor(log2 x) + 1.
 * Annotation ids: 0 serial, 1 unrolled, 2 unrolled explicitly, 3/4/5
 * blockIdx.x/y/z, 6/7/8 threadIdx.x/y/z, 9 vthread, 10 vectorized (the
 * annotated templates; 11, parallel, never occurs); a serial loop is unrolled when
 * auto_unroll_max_step > 0 and its sub-nest has at most that many
 * iterations.  Touch counts are distinct elements of the (padded) buffer
 * touched by the sub-nest rooted at the loop; reuse ratio is
 * floor(bottom-up / touch count); stride is the change of the buffer's flat
 * index for one step of the loop variable.
 * cfgs: device [n] uint64; feats: device [n][n_features] int32.
 * A single space only (not a set).  Rows whose index is >= n_configs are
 * filled with -1 and counted; at_space_errors() reports the count.
 * n == 0 is a no-op. */
at_status at_extract_features(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                              at_stream_t stream);

/* Full feature rows of Appendix A.2: per loop (outer to inner)
 * bitlen(length), annotation id, bitlen(top-down), bitlen(bottom-up), then
 * for each buffer bitlen(touch count), bitlen(reuse ratio), bitlen(stride):
 * 13 int32 per loop, n_loops * 13 per row (GEMM 130, conv2d 208).  Top-down
 * is the product of the lengths of the loops strictly outside the loop (1
 * for the outermost), bottom-up that of the loop and the loops inside it;
 * the other columns are those of at_extract_features.  cfgs: device [n]
 * uint64; feats: device [n][n_loops * 13] int32.  A single space only.
 * Out-of-range indices fill their row with -1 and are counted as for
 * at_extract_features.  n == 0 is a no-op. */
at_status at_extract_features_full(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                   at_stream_t stream);

/* The loop-context table of Appendix A.2 with its annotation column one-hot,
 * as the paper lists it: per loop (outer to inner) bitlen(length), 12
 * annotation columns (column h is 1 when the loop's annotation id is h, ids
 * as for at_extract_features, 0 otherwise), bitlen(top-down),
 * bitlen(bottom-up), then for each buffer bitlen(touch count), bitlen(reuse
 * ratio), bitlen(stride): 24 int32 per loop, n_loops * 24 per row (GEMM 240,
 * conv2d 384).  cfgs: device [n] uint64; feats: device [n][n_loops * 24]
 * int32.  A single space only.  Out-of-range indices fill their row with -1
 * and are counted as for at_extract_features.  n == 0 is a no-op. */
at_status at_extract_features_onehot(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                     at_stream_t stream);

/* Number of out-of-range configuration indices seen by at_extract_features
 * since the last call (synchronises the device; resets the counter). */
at_status at_space_errors(at_space_t space, uint64_t* n_out_of_range);

/* Gradient-boosted tree cost model f-hat (Section 3.1): n_trees full
 * binary trees of the given depth in heap order (node n has children 2n+1,
 * taken when x[fid[n]] < thr[n], and 2n+2).
 * fid, thr: host [n_trees][2^depth - 1] uint8 (fid < n_features);
 * leaf: host [n_trees][2^depth] float.  1 <= depth <= 12,
 * 1 <= n_features <= 256.  The tables are packed and uploaded to the
 * current device.  Synchronous. */
at_status at_ensemble_create(int n_trees, int depth, int n_features, const uint8_t* fid,
                             const uint8_t* thr, const float* leaf, at_ensemble_t* out);
void at_ensemble_destroy(at_ensemble_t ens);

/* Trained trees of any shape (Section 3.1: the cost model is a gradient-
 * boosted tree ensemble as a boosting library trains it; such trees are
 * neither full nor of one depth), given as node lists on the host: tree t
 * owns nodes tree_offsets[t] .. tree_offsets[t+1]-1 of the arrays, its root
 * first, and child indices count from the tree's first node.  Node i is a
 * split when left[i] >= 0: a row with x[feature[i]] < threshold[i] goes to
 * left[i], any other to right[i].  Node i is a leaf worth value[i] when
 * left[i] < 0 (right, feature and threshold are then ignored).
 *
 * at_trees_depth: checks that the lists form binary trees (every child in
 * range, every node reached at most once from its root; AT_E_INVALID
 * otherwise) and writes the level of the deepest leaf (0 for a tree that is
 * a single leaf) to *depth.
 *
 * at_trees_pad: writes the full-tree tables of at_ensemble_create at the given
 * depth (the deepest leaf's or more, 1 .. 12): fid, thr [n_trees][2^depth-1],
 * leaf [n_trees][2^depth], caller-owned host arrays.  A leaf above the last
 * level becomes a split on feature 0 with threshold 255 whose subtrees both
 * end in copies of the leaf, so every row reaches the leaf's value.  A
 * threshold t becomes ceil(t) clamped to [0, 255] (0 for t <= 0, 255 above
 * 255): x < t and x < ceil(t) agree for every integer x, so each row reaches
 * the same leaf value as in the lists whenever its features lie in
 * [0, 254] (loop features and relation features do).  Leaf indices that
 * at_gbt_predict reports are those of the padded trees.  Errors:
 * AT_E_INVALID for bad lists, a split feature outside [0, n_features), a
 * NaN threshold or a leaf below `depth`; AT_E_UNSUPPORTED for depth or
 * n_features out of range.
 *
 * at_ensemble_import: at_trees_pad at the deepest leaf's depth (at least 1),
 * then at_ensemble_create.  AT_E_UNSUPPORTED when a leaf lies below level 12.
 * Synchronous. */
at_status at_trees_depth(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                         int* depth);
at_status at_trees_pad(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                       const int32_t* feature, const float* threshold, const float* value, int n_features, int depth,
                       uint8_t* fid, uint8_t* thr, float* leaf);
at_status at_ensemble_import(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                             const int32_t* feature, const float* threshold, const float* value, int n_features,
                             at_ensemble_t* out);

/* Scores of n feature rows: the fp32 sum of each tree's reached leaf,
 * added in tree order starting from +0.0f (higher is better).
 * feats: device [n][n_features] int32 with values in [0, 255] (values
 * outside are clamped); scores: device [n] float; leaves: device
 * [n][n_trees] uint16 leaf indices, or NULL.  n == 0 is a no-op. */
at_status at_gbt_predict(at_ensemble_t ens, const int32_t* feats, int64_t n, float* scores,
                         uint16_t* leaves, at_stream_t stream);

/* Transfer model of Section 4, Eq. 4: f_hat(x) = f_hat_global(x) +
 * f_hat_local(x).  Each model's prediction is its own fp32 left fold over its
 * trees (as at_gbt_predict); scores[i] = fp32(global_i + local_i), global
 * first.  The two models may read different feature rows, for instance the
 * invariant context relation features for the global model and the loop
 * features for the local one.  feats_global: device [n][F_global] int32;
 * feats_local: device [n][F_local] int32; scores: device [n] float.
 * Enqueued on `stream` (two launches). */
at_status at_gbt_predict_global_local(at_ensemble_t global, const int32_t* feats_global, at_ensemble_t local,
                                      const int32_t* feats_local, int64_t n, float* scores, at_stream_t stream);

/* Persistent state of n_chains Markov chains (Section 3.3: chain states
 * persist across model updates): current knob values and score, absolute
 * step counter and a best list of the topk highest-scoring distinct
 * configurations seen.  Global chain ids are chain0 .. chain0+n_chains-1;
 * they key the chains' random streams, so a chain's trajectory does not
 * depend on which other chains run beside it.  For a space set, n_chains
 * must equal the set's last chain offset.  1 <= topk <= 64.  The chains
 * are initialised by the first at_sa_run: each knob value uniform over its
 * range, scored once and offered to the best list.  Synchronous. */
at_status at_chains_create(at_space_t space, int64_t chain0, int64_t n_chains, int topk,
                           uint64_t seed, at_chains_t* out);
void at_chains_destroy(at_chains_t chains);

/* Absolute step counter of the chains (the step_base of the next run). */
at_status at_chains_step(at_chains_t chains, uint64_t* step_abs);

/* Acceptance thresholds of simulated annealing with the model score as
 * energy (Section 3.3; the acceptance rule of Algorithm 1's search):
 * Metropolis thresholds for the next `steps` steps of chains
 * chain0 .. chain0+n_chains-1 starting at absolute step step_base:
 * thr[c][s] = fp32(T_s * ln(u)) computed in double, with
 * T_s = 1 - s/(steps-1) (T = 0 when steps == 1) and u = (r2 + 0.5) / 2^32,
 * r2 the third word of the Philox-4x32-10 block keyed by seed at counter
 * (chain, step_base + s, 0, 0).  A move of score change d (fp32) is then
 * accepted iff d >= thr, i.e. with probability min(1, exp(d / T_s)).
 * thr: host [n_chains][steps] float, caller-owned.  AT_E_INVALID for
 * steps < 1, a negative chain0 or n_chains, or a NULL thr with chains to
 * fill.  Runs on the host; nothing is enqueued. */
at_status at_sa_thresholds(uint64_t seed, int64_t chain0, int64_t n_chains, uint64_t step_base,
                           int steps, float* thr);

/* Runs `steps` annealing steps on every chain (Section 3.3, Algorithm 1's
 * inner search).  Per chain and step: draw the Philox block (chain,
 * step_abs, 0, 0); change one knob chosen uniformly among knobs with at
 * least two values to a uniformly chosen different value; extract the
 * candidate's features; score it with the ensemble; offer it to the best
 * list (ordered by score descending, then index ascending; duplicates are
 * skipped); accept it iff fp32(score - current) >= thr[c][s].
 * thr: device [n_chains][steps] float; best: device [n_chains][topk]
 * at_entry receiving a copy of the best lists after the run (entries with
 * flag 0 are empty).  The ensemble's feature count must match the space's
 * (AT_E_MISMATCH).  steps == 0 only initialises.
 * Two execution paths compute the same result bit for bit (at_sa_path):
 * chain-local, one launch per run in which each workgroup keeps a few chains
 * and streams the ensemble through its LDS every step, and tree-partitioned,
 * two launches per step in which workgroups hold disjoint tree groups and
 * exchange features and leaf values through global memory.  By default the
 * library takes the chain-local path when one workgroup keeps the whole
 * ensemble in its LDS or streams at most 768 KB of it per step, else the
 * tree-partitioned one.
 * Workspace: the first run on a chains handle, and any run with more trees
 * than before, allocates the chains' device workspace (tree-partitioned:
 * about n_chains * (16 * ceil(n_trees / 4) + 4 * ceil(n_features / 4) + 32)
 * bytes; chain-local: 16 bytes per chain), which synchronises the device;
 * later runs allocate nothing. */
at_status at_sa_run(at_space_t space, at_ensemble_t ens, at_chains_t chains, int steps,
                    const float* thr, at_entry* best, at_stream_t stream);

/* at_sa_run that also records, per chain and step, the proposed
 * configuration, its score and whether it was accepted.
 * trace: device [n_chains][steps] at_entry. */
at_status at_sa_run_traced(at_space_t space, at_ensemble_t ens, at_chains_t chains, int steps,
                           const float* thr, at_entry* best, at_entry* trace, at_stream_t stream);

/* at_sa_run whose energy is the transfer model of Section 4, Eq. 4:
 * f_hat(x) = f_hat_global(x) + f_hat_local(x).  The global model reads a
 * candidate's context relation features (the invariant representation, as
 * at_extract_relation_features writes them: 192 per configuration; its
 * ensemble must have n_features == 192, else AT_E_MISMATCH); the local model
 * reads its loop-context features (n_features of the space).  Each model's
 * prediction is its own fp32 left fold over its trees from +0.0f; a
 * candidate's score is fp32(global + local), the global one first.  Every
 * other step is at_sa_run's.  The chains keep the scores of the model that
 * scored them.  trace: device [n_chains][steps] at_entry, or NULL.  These runs
 * take the tree-partitioned path (two tree-kernel launches per step, one per
 * model): at_chains_set_path(AT_SA_PATH_LOCAL) makes them fail with
 * AT_E_UNSUPPORTED.  Workspace as at_sa_run, plus about n_chains *
 * (16 * ceil(global trees / 4) + 192) bytes on the first such run. */
at_status at_sa_run_global_local(at_space_t space, at_ensemble_t global, at_ensemble_t local, at_chains_t chains,
                                 int steps, const float* thr, at_entry* best, at_entry* trace,
                                 at_stream_t stream);

/* Context relation features (Section 4, "Context Relation Features for
 * GBT"; Appendix A.2 "Relation Feature") of n configurations: the invariant
 * representation the paper transfers across workloads.  Over the loops of
 * the nest (a single chain here), with thresholds beta_t = 2^t, t = 1..32,
 * per buffer b: R[0][b][t-1] = max over loops touching fewer than 2^t
 * elements of b of bitlen(reuse ratio), R[1][b][t-1] = max over the same
 * loops of bitlen(top-down), top-down being the product of the lengths of
 * the loops outside; 0 when no loop qualifies.
 * cfgs: device [n] uint64; feats: device [n][192] int32 row-major, buffers
 * in the loop features' order, 16-byte aligned.  A configuration index
 * outside [0, n_configs) gives a row of -1 and is counted as in
 * at_extract_features.  Enqueued on `stream`. */
at_status at_extract_relation_features(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                       at_stream_t stream);

/* Picks the batch of configurations to measure next (Algorithm 1 after the
 * annealing; Section 3.3, Eq. 3, and the epsilon-greedy step).
 * Q is the set of distinct configurations among the valid entries of cand;
 * its `pool` best (score descending, then index ascending; the paper's top
 * lambda*b) form the candidate set.  A greedy maximisation of
 *   L(S) = sum_{s in S} score(s) + alpha * sum_j |{ s_j : s in S }|
 * (score = -f_hat; s_j the value of knob j) then picks n_greedy of them one
 * at a time, each maximising its marginal gain score(s) + alpha * (number of
 * knobs whose value no earlier pick has), evaluated in fp32 as one product
 * and one sum, ties going to the earlier candidate in pool order.  Last,
 * n_random configurations are drawn uniformly among those of the space not
 * selected yet: draw i takes Philox-4x32-10 block (i, 0, 5, 0) keyed by
 * seed, u = r1 * 2^32 + r0, and the floor(u * remaining / 2^64)-th
 * unselected index in ascending order.
 * cand: device [n_cand] at_entry, for example the best lists written by
 * at_sa_run ([n_chains][topk]); the index of a valid entry must lie below
 * the space's configuration count (spaces hold fewer than 2^32), and an
 * index listed more than once must carry the same score each time (as best
 * lists do).  out: device
 * [n_greedy + n_random] at_entry: the greedy picks (flag 1) in pick order,
 * then the random ones (flag 2, score 0); slots left over when the pool or
 * the space runs out have flag 0.
 * Limits: 0 <= pool <= 1024, n_greedy + n_random <= 2048, a single space
 * (not a set) whose knobs have at most 65536 values each; AT_E_INVALID or
 * AT_E_UNSUPPORTED otherwise.  Enqueued on `stream`.  More than 2048
 * candidates use stream-ordered device scratch for a partial reduction:
 * 32 * ceil(n_cand / 2048) * P bytes, P the power of two at or above
 * max(pool, 1) (512 KiB for 262144 candidates at pool 128), taken with
 * hipMallocFromPoolAsync from a memory pool that the library creates on the
 * device.  The library keeps that scratch for the next such call on the
 * device (growing it when a call needs more) until the process ends, with
 * an event recorded after each call's kernels: a call makes its stream wait
 * for the previous call's event, so calls on different streams take their
 * turns on the scratch. */
at_status at_select_batch(at_space_t space, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                          float alpha, int n_random, uint64_t seed, at_entry* out, at_stream_t stream);

/* at_select_batch for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and the same result, bit for bit, with the
 * partial reduction of more than 2048 candidates kept in a fixed scratch
 * array that the library holds on each device until the process ends (two
 * buffers of 131072 entries, 4 MiB; looked up with hipGetSymbolAddress on
 * the first call on a device).  The call allocates and frees nothing.
 * Limit: ceil(n_cand / 2048) * P <= 131072, P the power of two at or above
 * max(pool, 1) (for example up to 262144 candidates at pool 1024, 2097152
 * at pool 128), AT_E_UNSUPPORTED beyond it; the other arguments and errors
 * are those of at_select_batch.
 * Every call on a device shares that device's scratch: calls that overlap
 * on one device (other streams, other threads) race and must be ordered by
 * the caller.  Nothing in the scratch needs to start at zero: each call
 * writes every entry it reads. */
at_status at_select_batch_noalloc(at_space_t space, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                                  float alpha, int n_random, uint64_t seed, at_entry* out, at_stream_t stream);

/* Execution path of the annealing runs of a chains handle. */
typedef enum {
    AT_SA_PATH_AUTO = 0,   /* chosen per run from the ensemble and chain count */
    AT_SA_PATH_TREES = 1,  /* tree-partitioned: two kernels per step */
    AT_SA_PATH_LOCAL = 2   /* chain-local: one persistent kernel per run */
} at_sa_path;

/* Selects the path of later runs on `chains` (AT_E_INVALID for an unknown
 * value).  A run asked to take the chain-local path when its plan does not
 * fit one workgroup's LDS fails with AT_E_UNSUPPORTED.  Either path may
 * continue chains the other has advanced. */
at_status at_chains_set_path(at_chains_t chains, int path);

/* The path the last run on `chains` took (AT_SA_PATH_AUTO before any run). */
at_status at_chains_last_path(at_chains_t chains, int* path);

/* Launch plan of the last run (measurement aid; read at_chains_last_path
 * to know which layout applies; zeros before any run).
 * Chain-local run: info[0] chains per workgroup, [1] threads per workgroup,
 * [2] workgroups, [3] trees per chunk, [4] chunks streamed per step (0:
 * nothing is streamed), [5] how leaves are reached: 0 from LDS (whole trees
 * resident or streamed), 1 streamed node blocks with leaves read from
 * global memory, 2 tree tops resident in LDS with the last level and its
 * leaves read from global memory, [6] dynamic LDS bytes, [7] bytes one
 * workgroup reads per step from outside its LDS.
 * Tree-partitioned run: info[0] trees per tree-kernel workgroup, [1] waves
 * per tree-kernel workgroup, [2] tree-kernel workgroups, [3] chain slices
 * per tree group, [4] 64-chain blocks per slice (a wave walks more than one
 * block when this exceeds [1]), [5] chain-kernel workgroups, [6] quads (4
 * features) per chain in a feature tile: the loop-context features that are
 * not constant over the space (set), when dropping the constant ones saves a
 * quad, [7] bytes of leaf values written and read back per step. */
at_status at_chains_last_plan(at_chains_t chains, int64_t info[8]);

/* Copies the chains' current configuration indices (device [n_chains]
 * uint64) and scores (device [n_chains] float); either may be NULL. */
at_status at_chains_export(at_chains_t chains, uint64_t* cur_cfg, float* cur_score,
                           at_stream_t stream);

/* Measurement aid.  With profiling enabled, at_sa_run and at_sa_run_traced
 * attach start/stop events to every launch of the annealing kernels (the
 * tree kernel, which walks the ensemble, and the chain kernel, which folds,
 * offers, accepts, proposes and featurises; the chain-local path's single
 * kernel counts as a tree kernel); results are unchanged.  The events are
 * created on first use and kept with the chains. */
at_status at_sa_set_profiling(at_chains_t chains, int enable);

/* Device time of the launches of the last profiled run: summed milliseconds
 * and launch counts of the tree and chain kernels; any output may be NULL.
 * Waits for the run to finish.  A run without profiling reports zeros. */
at_status at_sa_kernel_times(at_chains_t chains, double* tree_ms, int64_t* tree_launches, double* chain_ms,
                             int64_t* chain_launches);

/* Thread-local description of the last non-OK status ("" if none). */
const char* at_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* AUTOTENSOR_H */
