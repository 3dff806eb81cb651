// Picking the batch to measure after the annealing (Algorithm 1; Section
// 3.3, Eq. 3).
//
// Q is the set of distinct configurations in the chains' best lists.  The
// `pool` best of Q (score descending, then index ascending) form the
// candidate set (the paper's top lambda*b); a greedy submodular
// maximisation of
//     L(S) = sum_{s in S} score(s) + alpha * sum_j |{ s_j : s in S }|
// picks n_greedy of them, each pick maximising the marginal gain
// score(s) + alpha * (number of knobs whose value s adds to the picks)
// (fp32: one product, one sum; ties to the earlier candidate).  Then
// epsilon-greedy: n_random configurations uniform among those not selected
// yet, draw i from Philox block (i, 0, 5, 0): u = r1 * 2^32 + r0, the
// floor(u * remaining / 2^64)-th unselected index.
//
// k_reduce: each workgroup takes a slice of up to CHUNK candidates and
// writes its `keep` best distinct (score descending, index ascending,
// an index equal to its predecessor's in that order dropped) as a run of
// the power of two at or above keep (empty slots after them).  Best lists
// repeat configurations many times over and only the few best of a slice
// can reach its result, so the slice is not ordered whole:
//  1. exact repeats (the same 64-bit order key: score order bits, index)
//     are dropped, the first in entry order kept: they would be neighbours
//     once ordered, the first one first.  An LDS hash table holds the keys
//     and, per key, the smallest entry position;
//  2. a histogram of the remaining records' score order bits (scaled into
//     NBINS bins over their range: a bin is a range of order bits) gives the
//     smallest bin b whose bins up to b hold `keep` records;
//  3. the records up to bin b (a prefix of the ordered sequence) are
//     ordered, by counting (a record's place is the number of keys below
//     it) or for large sets by a merge sort, and the distinct ones taken;
//  4. should fewer than keep come out (the same index with different
//     scores, dropped as a neighbour's repeat) while records are left, the
//     prefix grows and 2-3 run again.
// Levels repeat until at most FINAL_MAX candidates remain.
// k_select (one workgroup): takes the pool from those the same way and
// decodes its knob values; then wave 0 alone runs the greedy
// rounds, each lane looking after pool candidates lane, lane + 64, ...: a
// round is a wave-wide arg-max of the gains (DPP steps, no workgroup
// barrier), then every lane clears the knobs the winner covers in its
// candidates' masks (and computes again the gains of the candidates whose
// masks changed).  The wave then ranks the picks in parallel (ascending
// indices) and makes each random draw with one wave-wide count: with S the
// picks in ascending order, the floor(u * remaining / 2^64) = k-th
// unselected index is k + j, j the number of positions i with
// S[i] - i <= k.
#include <mutex>

#include "at_chain.h"

namespace at {
namespace {

using namespace dev;

constexpr int SEL_WG = 1024;     // threads of both kernels
constexpr int CHUNK = 2048;      // candidates one reduction workgroup takes
constexpr int FINAL_MAX = 2048;  // candidates the final workgroup takes
constexpr int POOL_MAX = 1024;
constexpr int PICK_MAX = 2048;   // greedy plus random picks
constexpr int PER = FINAL_MAX / SEL_WG;   // records a thread holds in the pool stage
static_assert(CHUNK == FINAL_MAX && PER * SEL_WG == FINAL_MAX, "both kernels take the same slice size");
constexpr int HASH_LOG2 = 12;
constexpr int HASH_SLOTS = 1 << HASH_LOG2;   // exact-key table: at most half full
constexpr int NBINS_LOG2 = 11;
constexpr int NBINS = 1 << NBINS_LOG2;       // score histogram
static_assert(NBINS == 2 * SEL_WG, "the bin scan takes two bins a thread");
constexpr int RANK_MAX = SEL_WG;             // prefixes up to this size are ordered by counting
constexpr int RED_WORDS = 3 * (SEL_WG / 64) + 2;

// A candidate while it is ordered: a 64-bit order key, the score's order
// bits (smaller for a higher score, -0.0 as +0.0) in the high half and the
// configuration index in the low half (indices fit 32 bits: a space holds
// fewer than 2^32 configurations), ~0 for an empty slot; the score's own
// bits travel beside it in a second array.  Orderings compare the keys
// only (8-byte LDS reads).
constexpr uint64_t KEY_EMPTY = ~0ull;

struct RecBuf {
    uint64_t* key;
    uint32_t* bits;
};

// The record of entry e, or an empty one when e is not valid or not here
// (no branches, so that the loads that feed it are all in flight first).
__device__ __forceinline__ void rec_bits(const at_entry& e, bool here, uint64_t& key, uint32_t& bits) {
    const bool valid = here && e.flag != 0u;
    uint32_t b = __float_as_uint(e.score);
    const uint32_t z = b == 0x80000000u ? 0u : b;
    const uint32_t asc = (z & 0x80000000u) ? ~z : (z | 0x80000000u);
    key = valid ? (((uint64_t)~asc << 32) | (uint32_t)e.cfg) : KEY_EMPTY;
    bits = valid ? b : 0u;
}

__device__ __forceinline__ at_entry entry_of(uint64_t key, uint32_t bits) {
    at_entry e;
    e.cfg = (uint32_t)key;
    e.score = __uint_as_float(bits);
    e.flag = 1u;
    return e;
}

__device__ __forceinline__ at_entry empty_entry() {
    at_entry z;
    z.cfg = 0;
    z.score = 0.0f;
    z.flag = 0u;
    return z;
}

// Wave-wide primitives on DPP lane moves (no LDS round trip): a row
// shift or broadcast of x, lanes without a source taking 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_move(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xf, true);
}

// Largest unsigned value of the wave, in every lane: shifts within rows of
// 16, then row broadcasts, leave the maximum in lane 63 (a lane with no
// source takes 0, which never wins).
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    uint32_t o;
    o = dpp_move<0x111, 0xf>(x); x = o > x ? o : x;   // row_shr:1
    o = dpp_move<0x112, 0xf>(x); x = o > x ? o : x;   // row_shr:2
    o = dpp_move<0x114, 0xf>(x); x = o > x ? o : x;   // row_shr:4
    o = dpp_move<0x118, 0xf>(x); x = o > x ? o : x;   // row_shr:8
    o = dpp_move<0x142, 0xa>(x); x = o > x ? o : x;   // row_bcast:15 into rows 1 and 3
    o = dpp_move<0x143, 0xc>(x); x = o > x ? o : x;   // row_bcast:31 into rows 2 and 3
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// Inclusive prefix sum over the wave's lanes (the same steps with adds:
// after the row shifts a lane holds the sum of its row up to it, the row
// broadcasts add the rows before).
__device__ __forceinline__ uint32_t wave_inclusive_add(uint32_t x) {
    x += dpp_move<0x111, 0xf>(x);
    x += dpp_move<0x112, 0xf>(x);
    x += dpp_move<0x114, 0xf>(x);
    x += dpp_move<0x118, 0xf>(x);
    x += dpp_move<0x142, 0xa>(x);
    x += dpp_move<0x143, 0xc>(x);
    return x;
}

__device__ __forceinline__ int wave_sum(int x) {
    return __builtin_amdgcn_readlane((int)wave_inclusive_add((uint32_t)x), 63);
}

// Orders n records (a power of two) ascending, moving them between the LDS
// buffers a and b; returns the buffer that holds the result.  All threads
// call.  A level merges pairs of ascending runs of length L: every record
// finds its place in the merged run by a binary search of the partner run
// (a record of the left run counts the partner's records below it, one of
// the right run also those equal to it, so places are distinct).  A thread
// takes records tid, tid + blockDim.x, ...; the binary searches of its
// records go step by step together, so their LDS reads overlap.
__device__ RecBuf merge_sort(RecBuf a, RecBuf b, int n) {
    const int nt = (int)blockDim.x;
    RecBuf src = a, dst = b;
    int lg = 0;   // log2(L)
    for (int L = 1; L < n; L <<= 1, ++lg) {
        __syncthreads();   // the last level's records are in place
        uint64_t x[PER];
        uint32_t xb[PER];
        int base[PER], own[PER], cnt[PER];
        bool left[PER], here[PER];
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            const int i = (int)threadIdx.x + e * nt;
            here[e] = i < n;
            const int ii = here[e] ? i : 0;
            x[e] = src.key[ii];
            xb[e] = src.bits[ii];
            const int blk = ii >> (lg + 1);
            const int pos = ii & (2 * L - 1);
            left[e] = pos < L;
            own[e] = left[e] ? pos : pos - L;
            base[e] = blk * 2 * L + (left[e] ? L : 0);   // the partner run
            cnt[e] = 0;
        }
        // branch-free steps: every probe loads (clamped into the run), so
        // the PER loads of a step issue together
        for (int step = L; step > 0; step >>= 1) {
            uint64_t y[PER];
            int t[PER];
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                t[e] = cnt[e] + step;
                y[e] = src.key[base[e] + (t[e] <= L ? t[e] : L) - 1];
            }
#pragma unroll
            for (int e = 0; e < PER; ++e) {
                const bool before = left[e] ? y[e] < x[e] : y[e] <= x[e];
                cnt[e] = (t[e] <= L && before) ? t[e] : cnt[e];
            }
        }
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            if (here[e]) {
                const int blk0 = base[e] - (left[e] ? L : 0);
                dst.key[blk0 + own[e] + cnt[e]] = x[e];
                dst.bits[blk0 + own[e] + cnt[e]] = xb[e];
            }
        }
        const RecBuf t = src;
        src = dst;
        dst = t;
    }
    __syncthreads();
    return src;
}

// Orders the c distinct keys of src[0..c) (c <= SEL_WG) into dst[0..c) by
// counting: g threads look after a record (g = SEL_WG / the power of two
// at or above c, at most 64), each counting the keys below it in every
// g-th position, and the record goes to the sum.  All threads call.
__device__ void rank_sort(RecBuf src, RecBuf dst, int c) {
    int c2 = 1;
    while (c2 < c) c2 <<= 1;
    int g = SEL_WG / c2;
    g = g > 64 ? 64 : g;
    const int r = (int)threadIdx.x / g, p = (int)threadIdx.x & (g - 1);
    const bool mine = r < c;
    const uint64_t xr = src.key[mine ? r : 0];
    int cnt = 0;
    if (mine) {
        int j = p;
        // eight reads in flight, then their compares
        for (; j + 7 * g < c; j += 8 * g) {
            uint64_t y[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) y[u] = src.key[j + u * g];
#pragma unroll
            for (int u = 0; u < 8; ++u) cnt += y[u] < xr ? 1 : 0;
        }
        for (; j < c; j += g) cnt += src.key[j] < xr ? 1 : 0;
    }
    for (int off = 1; off < g; off <<= 1) cnt += __shfl_xor(cnt, off);
    if (mine && p == 0) {
        dst.key[cnt] = xr;
        dst.bits[cnt] = src.bits[r];
    }
    __syncthreads();
}

// Exclusive prefix sum of x over the block's threads (thread order); the
// total goes to *total.  All threads call; wsum has a slot per wave.
__device__ __forceinline__ int block_exclusive_scan(int x, int* wsum, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int inc = (int)wave_inclusive_add((uint32_t)x);
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    int before = 0, all = 0;
    for (int w = 0; w < nw; ++w) {
        const int t = wsum[w];
        before += w < wave ? t : 0;
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + inc - x;
}

// Ordered records v[0..n): the first `keep` distinct valid ones (an index
// equal to its predecessor's is dropped) go to out[0..keep), empty entries
// fill out[keep..slots); returns how many were found (at most keep).
// Thread t looks after the consecutive records [t * per, (t + 1) * per).
// All threads call.
__device__ int compact_distinct(RecBuf v, int n, at_entry* out, int keep, int slots, int* wsum) {
    const int nt = (int)blockDim.x;
    const int per = n > nt ? n / nt : 1;
    const int lo = threadIdx.x * per;
    auto fresh = [&](int i) {
        return v.key[i] != KEY_EMPTY && (i == 0 || (uint32_t)v.key[i] != (uint32_t)v.key[i - 1]);
    };
    int cnt = 0;
    for (int i = lo; i < lo + per && i < n; ++i) cnt += fresh(i) ? 1 : 0;
    int total = 0;
    int pos = block_exclusive_scan(cnt, wsum, &total);
    for (int i = lo; i < lo + per && i < n; ++i) {
        if (fresh(i)) {
            if (pos < keep) out[pos] = entry_of(v.key[i], v.bits[i]);
            ++pos;
        }
    }
    const int have = total < keep ? total : keep;
    for (int i = have + (int)threadIdx.x; i < slots; i += nt) out[i] = empty_entry();
    __syncthreads();
    return have;
}

// LDS of the pool stage.  The hash table (keys, first positions) lies over
// the two record buffers, which are written only once the table is done.
struct PoolLds {
    RecBuf v, w;        // [FINAL_MAX] each
    uint64_t* hkey;     // [HASH_SLOTS]
    uint32_t* hfirst;   // [HASH_SLOTS]
    uint32_t* hist;     // [NBINS]
    int* wsum;          // [SEL_WG / 64]
    uint32_t* red;      // [RED_WORDS]
};
constexpr size_t POOL_REGION_BYTES = (size_t)FINAL_MAX * (8 + 4) * 2;
static_assert((size_t)HASH_SLOTS * (8 + 4) <= POOL_REGION_BYTES, "the table fits over the record buffers");

__device__ __forceinline__ PoolLds pool_lds(uint64_t* region, uint32_t* hist, int* wsum, uint32_t* red) {
    PoolLds s;
    s.v.key = region;
    s.w.key = region + FINAL_MAX;
    s.v.bits = reinterpret_cast<uint32_t*>(region + 2 * FINAL_MAX);
    s.w.bits = s.v.bits + FINAL_MAX;
    s.hkey = region;
    s.hfirst = reinterpret_cast<uint32_t*>(region + HASH_SLOTS);
    s.hist = hist;
    s.wsum = wsum;
    s.red = red;
    return s;
}

__device__ __forceinline__ uint32_t key_hash(uint64_t k) {
    return (((uint32_t)k * 0x9e3779b1u) ^ ((uint32_t)(k >> 32) * 0x85ebca6bu)) >> (32 - HASH_LOG2);
}

// The `keep` best distinct of entries [base, base + n) of src (n <=
// FINAL_MAX, entries past total empty) -> out[0..keep) in order, empty
// entries up to out[slots); returns how many were found.  All threads call
// (the steps are in the comment at the top of this file).
__device__ int top_distinct(const at_entry* __restrict__ src, int64_t base, int64_t total, int n, at_entry* out,
                            int keep, int slots, const PoolLds& s) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NW = SEL_WG / 64;
    if (keep <= 0) {
        for (int i = tid; i < slots; i += SEL_WG) out[i] = empty_entry();
        return 0;
    }
    uint64_t x[PER];
    uint32_t xb[PER];
    for (int i = tid; i < HASH_SLOTS; i += SEL_WG) {
        s.hkey[i] = KEY_EMPTY;
        s.hfirst[i] = 0xffffffffu;
    }
    for (int i = tid; i < NBINS; i += SEL_WG) s.hist[i] = 0u;
    // loads from valid addresses on every lane (no branch around a load),
    // records past the end made empty afterwards
    at_entry en[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) en[e] = empty_entry();
    if (total > 0) {
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            const int64_t i = base + tid + e * SEL_WG;
            en[e] = src[i < total ? i : total - 1];
        }
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int i = tid + e * SEL_WG;
        const bool here = i < n && base + i < total;
        rec_bits(en[e], here, x[e], xb[e]);
    }
    __syncthreads();
    // 1. exact repeats: linear probing from the key's hash; every copy of a
    // key lands on its slot, which keeps the smallest entry position
    uint32_t slot[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        slot[e] = 0u;
        if (x[e] != KEY_EMPTY) {
            uint32_t h = key_hash(x[e]);
            while (true) {
                const uint64_t prev = atomicCAS(&s.hkey[h], KEY_EMPTY, x[e]);
                if (prev == KEY_EMPTY || prev == x[e]) break;
                h = (h + 1u) & (HASH_SLOTS - 1u);
            }
            slot[e] = h;
            atomicMin(&s.hfirst[h], (uint32_t)(tid + e * SEL_WG));
        }
    }
    __syncthreads();
    bool kept[PER];
    uint32_t ob[PER];
    uint32_t mn = 0xffffffffu, mx = 0u, nk = 0u;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        kept[e] = x[e] != KEY_EMPTY && s.hfirst[slot[e]] == (uint32_t)(tid + e * SEL_WG);
        ob[e] = (uint32_t)(x[e] >> 32);
        if (kept[e]) {
            mn = ob[e] < mn ? ob[e] : mn;
            mx = ob[e] > mx ? ob[e] : mx;
            ++nk;
        }
    }
    mn = ~wave_max_u32(~mn);
    mx = wave_max_u32(mx);
    nk = (uint32_t)wave_sum((int)nk);
    if (lane == 0) {
        s.red[wave] = mn;
        s.red[NW + wave] = mx;
        s.red[2 * NW + wave] = nk;
    }
    __syncthreads();
    mn = 0xffffffffu;
    mx = 0u;
    nk = 0u;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        const uint32_t a = s.red[w], b = s.red[NW + w];
        mn = a < mn ? a : mn;
        mx = b > mx ? b : mx;
        nk += s.red[2 * NW + w];
    }
    if (nk == 0u) {
        for (int i = tid; i < slots; i += SEL_WG) out[i] = empty_entry();
        __syncthreads();
        return 0;
    }
    // 2. histogram: bin (ob - mn) >> sh < NBINS
    const uint32_t range = mx - mn;
    const int bits = range ? 32 - __clz((int)range) : 0;
    const int sh = bits > NBINS_LOG2 ? bits - NBINS_LOG2 : 0;
    uint32_t bin[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        bin[e] = (ob[e] - mn) >> sh;
        if (kept[e]) atomicAdd(&s.hist[bin[e]], 1u);
    }
    __syncthreads();
    const int h0 = (int)s.hist[2 * tid], h1 = (int)s.hist[2 * tid + 1];
    int all = 0;
    const int before = block_exclusive_scan(h0 + h1, s.wsum, &all);
    int target = keep < (int)nk ? keep : (int)nk;
    int have = 0;
    while (true) {
        // the smallest bin whose bins up to it hold `target` records
        if (before < target && target <= before + h0 + h1) {
            s.red[3 * NW] = before + h0 >= target ? 2u * tid : 2u * tid + 1u;
            s.red[3 * NW + 1] = 0u;
        }
        __syncthreads();
        const uint32_t last = s.red[3 * NW];
        // 3. the records up to that bin into w (in any order)
#pragma unroll
        for (int e = 0; e < PER; ++e) {
            const bool in = kept[e] && bin[e] <= last;
            const uint64_t bal = __ballot(in);
            uint32_t at = 0u;
            if (lane == 0 && bal) at = atomicAdd(&s.red[3 * NW + 1], (uint32_t)__popcll(bal));
            at = (uint32_t)__builtin_amdgcn_readfirstlane((int)at);
            if (in) {
                const uint32_t p = at + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
                s.w.key[p] = x[e];
                s.w.bits[p] = xb[e];
            }
        }
        __syncthreads();
        const int c = (int)s.red[3 * NW + 1];
        if (c <= RANK_MAX) {
            rank_sort(s.w, s.v, c);
            have = compact_distinct(s.v, c, out, keep, slots, s.wsum);
        } else {
            int c2 = 1;
            while (c2 < c) c2 <<= 1;
            for (int i = c + tid; i < c2; i += SEL_WG) s.w.key[i] = KEY_EMPTY;
            const RecBuf sorted = merge_sort(s.w, s.v, c2);
            have = compact_distinct(sorted, c2, out, keep, slots, s.wsum);
        }
        // 4. too few distinct while records are left: a longer prefix
        if (have >= keep || c >= (int)nk) break;
        target = c + 2 * (keep - have);
        target = target < (int)nk ? target : (int)nk;
    }
    return have;
}

// Workgroup b: entries [b * CHUNK, ...) of src -> its `keep` best distinct
// as the run dst + b * slots.
__global__ __launch_bounds__(SEL_WG) void k_reduce(const at_entry* __restrict__ src, int64_t n, int keep, int slots,
                                                   at_entry* __restrict__ dst) {
    __shared__ uint64_t region[POOL_REGION_BYTES / 8];
    __shared__ uint32_t hist[NBINS];
    __shared__ int wsum[SEL_WG / 64];
    __shared__ uint32_t red[RED_WORDS];
    const PoolLds s = pool_lds(region, hist, wsum, red);
    top_distinct(src, (int64_t)blockIdx.x * CHUNK, n, CHUNK, dst + (int64_t)blockIdx.x * slots, keep, slots, s);
}

struct SelectArgs {
    const SpaceDesc* desc;
    const at_entry* src;      // candidates, or partial results (at most FINAL_MAX)
    int64_t n;
    int pool;
    int n_greedy;
    float alpha;
    int n_random;
    uint64_t seed;
    at_entry* out;            // [n_greedy + n_random]
};

// Ascending order bits of a finite gain (-0.0 as +0.0).
// (g + 0.0f is g for every g but -0.0, which it turns into +0.0; a negative
// value's bits are all flipped, a positive value's sign bit set.)
__device__ __forceinline__ uint32_t gain_order(float g) {
    const uint32_t b = __float_as_uint(g + 0.0f);
    return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}

// The greedy rounds of wave 0 for up to 64 * CPL pool candidates; knob
// values of a lane's candidates (packed in pairs) are held in registers for
// up to 4 candidates a lane, read from LDS for more.  Each candidate's
// gain is kept as its order bits (0: picked or absent; every finite gain
// orders above 0) and computed again only in rounds that take knobs from
// some candidate (the winner usually adds no knob, so most rounds are just
// the arg-max).  A round takes the largest order bits over the wave, then
// the earliest candidate that has them: candidate lane + 64 i comes before
// every candidate of a later i, so the first i whose ballot is not empty,
// and its lowest lane, give the winner.  The winners' indices go to
// win_idx.
template <int CPL>
__device__ void greedy_rounds(const SelectArgs& a, const at_entry* pool, const uint32_t* vals, int have, int m,
                              int* win_idx, int rounds) {
    constexpr int W = MAX_KNOBS / 2;
    const int lane = threadIdx.x & 63;
    const uint32_t all = m >= 32 ? 0xffffffffu : (1u << m) - 1u;
    constexpr bool REG = CPL <= 4;
    constexpr int KR = REG ? CPL : 1;
    float sc[CPL];
    uint32_t fresh[CPL], go[CPL], kv[KR][W];
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
        const int c = lane + 64 * i;
        const bool mine = c < have;
        sc[i] = mine ? pool[c].score : 0.0f;
        fresh[i] = mine ? all : 0u;
        if constexpr (REG) {
#pragma unroll
            for (int j = 0; j < W; ++j) kv[i][j] = mine ? vals[c * W + j] : 0u;
        }
        go[i] = mine ? gain_order(sc[i] + a.alpha * (float)__popc(fresh[i])) : 0u;
    }
    int wins = 0;
    for (int r = 0; r < rounds; ++r) {
        uint32_t best = 0u;
#pragma unroll
        for (int i = 0; i < CPL; ++i) best = go[i] > best ? go[i] : best;
        best = wave_max_u32(best);
        // the first i whose ballot is not empty, and its lowest lane
        int wi = CPL - 1;
        uint64_t mw = __ballot(go[CPL - 1] == best);
#pragma unroll
        for (int i = CPL - 2; i >= 0; --i) {
            const uint64_t bal = __ballot(go[i] == best);
            if (bal) {
                wi = i;
                mw = bal;
            }
        }
        const int wl = (int)__builtin_ctzll(mw), win = 64 * wi + wl;
        // the knobs whose value the winner adds (its fresh knobs): only
        // candidates with the same value at those knobs lose them
        uint32_t wf = 0u;
#pragma unroll
        for (int i = 0; i < CPL; ++i)
            if (i == wi) wf = fresh[i];
        uint32_t added = (uint32_t)__builtin_amdgcn_readlane((int)wf, wl);
#pragma unroll
        for (int i = 0; i < CPL; ++i)
            if (i == wi && lane == wl) go[i] = 0u;
        if (added) {
            while (added) {
                const int j = __builtin_ctz(added);
                added &= added - 1u;
                const int jw = j >> 1, sh = 16 * (j & 1);
                uint32_t wv;
                if constexpr (REG) {
                    uint32_t x = 0u;
#pragma unroll
                    for (int i = 0; i < CPL; ++i)
                        if (i == wi) x = kv[i][jw];
                    wv = ((uint32_t)__builtin_amdgcn_readlane((int)x, wl) >> sh) & 0xffffu;
                } else {
                    wv = (vals[win * W + jw] >> sh) & 0xffffu;
                }
#pragma unroll
                for (int i = 0; i < CPL; ++i) {
                    const uint32_t mine = REG ? kv[REG ? i : 0][jw] : vals[(lane + 64 * i) * W + jw];
                    if (((mine >> sh) & 0xffffu) == wv) fresh[i] &= ~(1u << j);
                }
            }
#pragma unroll
            for (int i = 0; i < CPL; ++i)
                go[i] = go[i] ? gain_order(sc[i] + a.alpha * (float)__popc(fresh[i])) : 0u;
        }
        // lane r % 64 keeps the winner of round r, 64 rounds to a store
        wins = lane == (r & 63) ? win : wins;
        if ((r & 63) == 63 || r == rounds - 1)
            if ((r & ~63) + lane <= r) win_idx[(r & ~63) + lane] = wins;
    }
}

// Four waves per SIMD (the workgroup's sixteen): up to 128 VGPRs, so the
// greedy wave keeps its candidates in registers without spilling.
__global__ __launch_bounds__(SEL_WG) __attribute__((amdgpu_waves_per_eu(1, 4))) void k_select(SelectArgs a) {
    extern __shared__ uint4 sel_lds[];
    uint64_t* region = reinterpret_cast<uint64_t*>(sel_lds);                     // the pool stage's buffers
    at_entry* pool = reinterpret_cast<at_entry*>(region + POOL_REGION_BYTES / 8);   // [POOL_MAX]
    uint32_t* vals = reinterpret_cast<uint32_t*>(pool + POOL_MAX);               // [POOL_MAX][MAX_KNOBS / 2]
    // after the pool stage its buffers hold the picks
    uint64_t* picked = region;                                                   // [PICK_MAX], pick order
    uint64_t* sorted = picked + PICK_MAX;                                        // [PICK_MAX], ascending
    static_assert((size_t)PICK_MAX * 8 * 2 <= POOL_REGION_BYTES, "the picks fit the pool stage's buffers");
    __shared__ uint32_t hist[NBINS];
    __shared__ int wsum[SEL_WG / 64];
    __shared__ uint32_t red[RED_WORDS];
    const int tid = threadIdx.x, lane = tid & 63;
    const SpaceDesc& sd = *a.desc;

    // the pool: the `pool` best distinct candidates
    const int have = top_distinct(a.src, 0, a.n, (int)a.n, pool, a.pool, a.pool, pool_lds(region, hist, wsum, red));

    // knob values of the pool candidates, packed in pairs (knob j of
    // candidate c is 16-bit half c * MAX_KNOBS + j), a thread per knob:
    // value j of index x is floor(x / radix_j) mod size_j (indices fit 32
    // bits: a space has fewer than 2^32 configurations)
    const int m = sd.n_knobs;
    uint16_t* vals16 = reinterpret_cast<uint16_t*>(vals);
    for (int t = tid; t < have * MAX_KNOBS; t += SEL_WG) {
        const int c = t / MAX_KNOBS, j = t - c * MAX_KNOBS;
        uint32_t v = 0u;
        if (j < m) v = ((uint32_t)pool[c].cfg / (uint32_t)sd.radix[j]) % sd.knob_size[j];
        vals16[t] = (uint16_t)v;
    }
    __syncthreads();
    if (tid >= 64) return;   // the rounds and the draws are wave 0's; no barrier follows

    // the same in every lane; readfirstlane lets the compiler see it
    const int rounds = __builtin_amdgcn_readfirstlane(a.n_greedy < have ? a.n_greedy : have);
    const int cpl = (have + 63) / 64;
    int* win_idx = reinterpret_cast<int*>(sorted);   // free until the ranking below
    if (cpl <= 1) greedy_rounds<1>(a, pool, vals, have, m, win_idx, rounds);
    else if (cpl <= 2) greedy_rounds<2>(a, pool, vals, have, m, win_idx, rounds);
    else if (cpl <= 4) greedy_rounds<4>(a, pool, vals, have, m, win_idx, rounds);
    else if (cpl <= 8) greedy_rounds<8>(a, pool, vals, have, m, win_idx, rounds);
    else greedy_rounds<16>(a, pool, vals, have, m, win_idx, rounds);
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    // the picks out, in pick order
    for (int r = lane; r < rounds; r += 64) {
        at_entry e = pool[win_idx[r]];
        e.flag = 1u;
        a.out[r] = e;
        picked[r] = e.cfg;
    }

    // the picks in ascending order: pick i goes to its rank (picks are
    // distinct)
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    for (int i = lane; i < rounds; i += 64) {
        const uint64_t x = picked[i];
        int rank = 0, j = 0;
        // eight reads in flight, then their compares
        for (; j + 8 <= rounds; j += 8) {
            uint64_t y[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) y[u] = picked[j + u];
#pragma unroll
            for (int u = 0; u < 8; ++u) rank += y[u] < x ? 1 : 0;
        }
        for (; j < rounds; ++j) rank += picked[j] < x ? 1 : 0;
        sorted[rank] = x;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();

    // epsilon-greedy draws, then empty slots.  The draws' random words do
    // not depend on the picks: each lane makes one, 64 draws at a time.
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    int n_sel = rounds, slot = rounds;
    uint64_t u_lane = 0;
    auto draw_word = [&](int i) -> uint64_t {
        if ((i & 63) == 0 && i + lane < a.n_random) {
            const U4 r = philox(k0, k1, U4{(uint32_t)(i + lane), 0u, 5u, 0u});
            u_lane = ((uint64_t)r.y << 32) | r.x;
        }
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u_lane, i & 63);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u_lane >> 32), i & 63);
        return ((uint64_t)hi << 32) | lo;
    };
    auto put = [&](uint64_t cfg) {
        if (lane == 0) {
            at_entry e;
            e.cfg = cfg;
            e.score = 0.0f;
            e.flag = 2u;
            a.out[slot] = e;
        }
    };
    if (rounds + a.n_random <= 64) {
        // every selected index fits the wave: lane p holds sorted[p]
        uint64_t sv = lane < rounds ? sorted[lane] : ~0ull;
        for (int i = 0; i < a.n_random; ++i) {
            const uint64_t remaining = sd.n_configs - (uint64_t)n_sel;
            if (remaining == 0) break;
            const uint64_t k = __umul64hi(draw_word(i), remaining);
            // j = #{positions p with sorted[p] - p <= k}: those picks lie at
            // or below the drawn index, which is then k + j
            const int j = (int)__popcll(__ballot(lane < n_sel && sv - (uint64_t)lane <= k));
            const uint64_t cfg = k + (uint64_t)j;
            // insert at position j: lanes above it take their lower
            // neighbour's value (a wave shift right by one lane)
            const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)sv, 0x138, 0xf, 0xf, false);
            const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(sv >> 32), 0x138, 0xf, 0xf,
                                                                      false);
            const uint64_t below = ((uint64_t)hi << 32) | lo;
            sv = lane > j ? below : (lane == j ? cfg : sv);
            put(cfg);
            ++n_sel;
            ++slot;
        }
    } else {
        for (int i = 0; i < a.n_random; ++i) {
            const uint64_t remaining = sd.n_configs - (uint64_t)n_sel;
            if (remaining == 0) break;
            const uint64_t k = __umul64hi(draw_word(i), remaining);
            int j = 0;
            for (int p = lane; p < n_sel; p += 64) j += (sorted[p] - (uint64_t)p <= k) ? 1 : 0;
            j = wave_sum(j);
            const uint64_t cfg = k + (uint64_t)j;
            // insert at position j: the picks from j on move up by one, each
            // lane reading all of its picks before any lane writes
            for (int base = (n_sel - 1) & ~63; base >= 0; base -= 64) {
                const int p = base + lane;
                const uint64_t x = (p < n_sel) ? sorted[p] : 0;
                __builtin_amdgcn_s_waitcnt(0xc07f);
                __builtin_amdgcn_wave_barrier();
                if (p < n_sel && p >= j) sorted[p + 1] = x;
                __builtin_amdgcn_s_waitcnt(0xc07f);
                __builtin_amdgcn_wave_barrier();
            }
            if (lane == 0) sorted[j] = cfg;
            put(cfg);
            __builtin_amdgcn_s_waitcnt(0xc07f);
            __builtin_amdgcn_wave_barrier();
            ++n_sel;
            ++slot;
        }
    }
    for (int q = slot + lane; q < a.n_greedy + a.n_random; q += 64) a.out[q] = empty_entry();
}

size_t select_lds_bytes() {
    return POOL_REGION_BYTES + (size_t)POOL_MAX * sizeof(at_entry) + (size_t)POOL_MAX * (MAX_KNOBS / 2) * 4;
}

}  // namespace

int select_pool_max() { return POOL_MAX; }
int select_pick_max() { return PICK_MAX; }

// Slots of one reduction workgroup's result: the power of two at or above
// max(pool, 1), so that the results form whole ascending runs.
static int run_slots(int pool) {
    int r = 1;
    while (r < pool) r <<= 1;
    return r;
}

// Entries of each of the two partial-result buffers the reduction of n_cand
// candidates needs (0 when n_cand fits the final workgroup).
int64_t select_scratch_entries(int64_t n_cand, int pool) {
    if (n_cand <= FINAL_MAX) return 0;
    return (n_cand + CHUNK - 1) / CHUNK * run_slots(pool);
}

// Scratch of the entry point that allocates nothing: the two partial-result
// buffers, each SELECT_SCRATCH_ENTRIES entries (2 MiB), in one array per
// device that lives as long as the process.  Host code never passes the
// array's name to a kernel: the address comes from hipGetSymbolAddress,
// once per device.
constexpr int64_t SELECT_SCRATCH_ENTRIES = 131072;
static __device__ __align__(256) at_entry select_scratch[2 * SELECT_SCRATCH_ENTRIES];

int64_t select_scratch_max_entries() { return SELECT_SCRATCH_ENTRIES; }

hipError_t select_scratch_ptr(int device, at_entry** out) {
    constexpr int MAX_DEVICES = 64;
    static std::mutex mu;
    static at_entry* ptr[MAX_DEVICES] = {};
    if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[device]) {
        void* p = nullptr;
        // the caller has made `device` current
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(select_scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        ptr[device] = static_cast<at_entry*>(p);
    }
    *out = ptr[device];
    return hipSuccess;
}

// The allocating entry point's scratch comes from a memory pool of the
// library's own on each device, whose release threshold is unlimited:
// memory freed back to it stays reserved, so that later calls take it again
// without mapping new memory.  Created by the first call that needs scratch
// on the device (which is current), kept until the process ends.
static hipError_t select_mem_pool(int device, hipMemPool_t* out) {
    constexpr int MAX_DEVICES = 64;
    static std::mutex mu;
    static hipMemPool_t pools[MAX_DEVICES] = {};
    if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!pools[device]) {
        hipMemPoolProps props{};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = device;
        hipMemPool_t p = nullptr;
        hipError_t e = hipMemPoolCreate(&p, &props);
        if (e != hipSuccess) return e;
        uint64_t keep_all = UINT64_MAX;
        e = hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep_all);
        if (e != hipSuccess) {
            (void)hipMemPoolDestroy(p);
            return e;
        }
        pools[device] = p;
    }
    *out = pools[device];
    return hipSuccess;
}

// The allocating entry point keeps, on each device, the scratch of its
// last call that needed one (grown when a call needs more) and an event
// recorded after that call's kernels on the call's stream.  A call first
// makes its own stream wait for that event, so calls on any streams use
// (or free) the scratch one after the other.  Both live until the process
// ends.
struct SelectCache {
    at_entry* ptr = nullptr;
    int64_t entries = 0;
    hipEvent_t done = nullptr;
};

hipError_t launch_select(const at_space_s& sp, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                         float alpha, int n_random, uint64_t seed, at_entry* out, hipStream_t stream,
                         at_entry* scratch) {
    static bool configured = false;
    hipError_t e = hipSuccess;
    if (!configured) {
        e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_select), hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)select_lds_bytes());
        if (e != hipSuccess) return e;
        configured = true;
    }
    // reduce the candidates to at most FINAL_MAX entries: each level keeps
    // the `keep` best distinct of every CHUNK-entry slice as a run of `slots`
    // (half a slice or less)
    const int keep = pool > 0 ? pool : 1;
    const int slots = run_slots(pool);
    const at_entry* src = cand;
    int64_t n = n_cand;
    at_entry* bufs[2] = {nullptr, nullptr};
    const int64_t need = select_scratch_entries(n_cand, pool);
    const bool own = need > 0 && !scratch;   // scratch of our own (both buffers in one)
    static std::mutex cache_mu;
    static SelectCache caches[64];
    std::unique_lock<std::mutex> lock(cache_mu, std::defer_lock);   // held while the kernels are enqueued
    SelectCache* cache = nullptr;
    if (need > 0 && scratch) {
        if (need > SELECT_SCRATCH_ENTRIES) return hipErrorInvalidValue;
        bufs[0] = scratch;
        bufs[1] = scratch + SELECT_SCRATCH_ENTRIES;
    } else if (own) {
        if (sp.device < 0 || sp.device >= 64) return hipErrorInvalidDevice;
        lock.lock();
        cache = &caches[sp.device];
        // the event orders calls only (a later call's kernels overwrite what
        // an earlier call's kernels read), so it needs no system-scope fence
        if (!cache->done && (e = hipEventCreateWithFlags(&cache->done, hipEventDisableTiming |
                                                                           hipEventDisableSystemFence)) != hipSuccess) {
            cache->done = nullptr;
            return e;
        }
        // the last call's kernels are done with the scratch first
        if ((e = hipStreamWaitEvent(stream, cache->done, 0)) != hipSuccess) return e;
        if (cache->entries < 2 * need) {
            if (cache->ptr) (void)hipFreeAsync(cache->ptr, stream);
            cache->ptr = nullptr;
            cache->entries = 0;
            hipMemPool_t mp = nullptr;
            if ((e = select_mem_pool(sp.device, &mp)) != hipSuccess) return e;
            void* b = nullptr;
            if ((e = hipMallocFromPoolAsync(&b, 2 * (size_t)need * sizeof(at_entry), mp, stream)) != hipSuccess)
                return e;
            cache->ptr = static_cast<at_entry*>(b);
            cache->entries = 2 * need;
        }
        bufs[0] = cache->ptr;
        bufs[1] = cache->ptr + need;
    }
    int cur = 0;
    while (n > FINAL_MAX) {
        const int64_t groups = (n + CHUNK - 1) / CHUNK;
        hipLaunchKernelGGL(k_reduce, dim3((unsigned)groups), dim3(SEL_WG), 0, stream, src, n, keep, slots, bufs[cur]);
        if ((e = hipGetLastError()) != hipSuccess) break;
        src = bufs[cur];
        n = groups * slots;
        cur ^= 1;
    }
    if (e != hipSuccess) {
        if (own) (void)hipEventRecord(cache->done, stream);
        return e;
    }
    SelectArgs a{};
    a.desc = static_cast<const SpaceDesc*>(sp.d_descs.p);
    a.src = src;
    a.n = n;
    a.pool = pool;
    a.n_greedy = n_greedy;
    a.alpha = alpha;
    a.n_random = n_random;
    a.seed = seed;
    a.out = out;
    hipLaunchKernelGGL(k_select, dim3(1), dim3(SEL_WG), select_lds_bytes(), stream, a);
    e = hipGetLastError();
    if (own) {
        const hipError_t r = hipEventRecord(cache->done, stream);
        if (e == hipSuccess) e = r;
    }
    return e;
}

}  // namespace at
