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
// k_reduce: each workgroup orders a slice of up to CHUNK candidates in LDS
// (on 16-byte records that carry the score's order bits, the score itself
// and the index), drops repeated indices and writes its best `keep`
// candidates as a run of the power of two at or above keep (empty slots
// after them).  Ordering is a merge sort: at each level every record finds
// its place in the merged run by a binary search of the partner run (a
// record of the left run counts the partner's records that precede it, one
// of the right run also those equal to it, so places are distinct), one
// barrier per level.  Raw candidates are runs of one; a partial result from
// the level before is a slice of sorted runs, so later levels and the final
// workgroup start from longer runs.
// Levels repeat until at most FINAL_MAX candidates remain.
// k_select (one workgroup): orders and compacts those the same way into the
// pool and decodes its knob values; then wave 0 alone runs the greedy
// rounds, each lane looking after pool candidates lane, lane + 64, ...: a
// round is a wave-wide arg-max of the gains (DPP steps, no workgroup
// barrier), then every lane clears the knobs the winner covers in its
// candidates' masks.  The wave then ranks the picks in parallel (ascending
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
constexpr int CHUNK = 2048;      // candidates one reduction workgroup orders
constexpr int FINAL_MAX = 2048;  // candidates the final workgroup orders
constexpr int POOL_MAX = 1024;
constexpr int PICK_MAX = 2048;   // greedy plus random picks

// A candidate while it is ordered: a 64-bit order key, the score's order
// bits (smaller for a higher score, -0.0 as +0.0) in the high half and the
// configuration index in the low half (indices fit 32 bits: a space holds
// fewer than 2^32 configurations), ~0 for an empty slot; the score's own
// bits travel beside it in a second array.  Binary searches read the keys
// only (8-byte LDS reads).
constexpr uint64_t KEY_EMPTY = ~0ull;

struct RecBuf {
    uint64_t* key;
    uint32_t* bits;
};

__device__ __forceinline__ void rec_of(const at_entry& e, uint64_t& key, uint32_t& bits) {
    if (!e.flag) {
        key = KEY_EMPTY;
        bits = 0u;
        return;
    }
    bits = __float_as_uint(e.score);
    uint32_t b = bits;
    if (b == 0x80000000u) b = 0u;
    const uint32_t asc = (b & 0x80000000u) ? ~b : (b | 0x80000000u);   // ascending float order
    key = ((uint64_t)~asc << 32) | (uint32_t)e.cfg;
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

// Orders n records (a power of two) made of ascending runs of length run
// (a power of two, 1 for unordered input) ascending, moving them between
// the LDS buffers a and b; returns the buffer that holds the result.  All
// threads call.  A thread takes records tid, tid + blockDim.x, ...; the
// binary searches of its records go step by step together, so their LDS
// reads overlap.
// A level whose pairs of runs are already in order (the last record of
// every left run precedes or equals the first of its right run, so the
// merge would only concatenate them) is skipped, until the first level
// that is not: best lists arrive as ordered runs of the list length.
template <int PER>
__device__ RecBuf merge_sort(RecBuf a, RecBuf b, int n, int run) {
    const int nt = (int)blockDim.x;
    RecBuf src = a, dst = b;
    bool check = true;
    int lg = 0;   // log2(L)
    while ((1 << lg) < run) ++lg;
    for (int L = run; L < n; L <<= 1, ++lg) {
        __syncthreads();   // the last level's records are in place
        if (check) {
            int ordered = 1;
            for (int blk = (int)threadIdx.x; blk * 2 * L < n; blk += nt)
                ordered &= src.key[blk * 2 * L + L] < src.key[blk * 2 * L + L - 1] ? 0 : 1;
            if (__syncthreads_and(ordered)) continue;
            check = false;
        }
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
        // the PER loads of a step issue together.  A record of the left run
        // counts the partner's records below it, one of the right run also
        // those equal to it, so places are distinct.
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

// Exclusive prefix sum of x over the block's threads (thread order); the
// total goes to *total.  All threads call; wsum has a slot per wave.
__device__ __forceinline__ int block_exclusive_scan(int x, int* wsum, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int inc = x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
    }
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

// Records of entries [base, base + n) of src (empty past the end); all
// threads call.
__device__ __forceinline__ void load_slice(const at_entry* __restrict__ src, int64_t base, int64_t total, int n,
                                           RecBuf v) {
    for (int i = threadIdx.x; i < n; i += blockDim.x)
        rec_of(base + i < total ? src[base + i] : empty_entry(), v.key[i], v.bits[i]);
}

// Workgroup b: entries [b * CHUNK, ...) of src, ascending runs of length
// run -> its `keep` best distinct as the run dst + b * slots.
__global__ __launch_bounds__(SEL_WG) void k_reduce(const at_entry* __restrict__ src, int64_t n, int run, int keep,
                                                   int slots, at_entry* __restrict__ dst) {
    __shared__ uint64_t k0[CHUNK], k1[CHUNK];
    __shared__ uint32_t b0[CHUNK], b1[CHUNK];
    __shared__ int wsum[SEL_WG / 64];
    const RecBuf v{k0, b0}, w{k1, b1};
    load_slice(src, (int64_t)blockIdx.x * CHUNK, n, CHUNK, v);
    const RecBuf sorted = merge_sort<CHUNK / SEL_WG>(v, w, CHUNK, run);
    compact_distinct(sorted, CHUNK, dst + (int64_t)blockIdx.x * slots, keep, slots, wsum);
}

struct SelectArgs {
    const SpaceDesc* desc;
    const at_entry* src;      // candidates, or partial results (at most FINAL_MAX)
    int64_t n;
    int run;                  // ascending runs of src (1: unordered)
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

__device__ __forceinline__ int wave_sum(int x) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
    return x;
}

// Largest unsigned value of the wave, in every lane: DPP shifts within
// rows of 16, then row broadcasts, leave the maximum in lane 63 (a lane
// with no source takes 0, which never wins).
template <int CTRL, int ROWS>
__device__ __forceinline__ uint32_t dpp_max_step(uint32_t x) {
    const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xf, true);
    return o > x ? o : x;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = dpp_max_step<0x111, 0xf>(x);   // row_shr:1
    x = dpp_max_step<0x112, 0xf>(x);   // row_shr:2
    x = dpp_max_step<0x114, 0xf>(x);   // row_shr:4
    x = dpp_max_step<0x118, 0xf>(x);   // row_shr:8
    x = dpp_max_step<0x142, 0xa>(x);   // row_bcast:15 into rows 1 and 3
    x = dpp_max_step<0x143, 0xc>(x);   // row_bcast:31 into rows 2 and 3
    return (uint32_t)__builtin_amdgcn_readlane((int)x, 63);
}

// The greedy rounds of wave 0 for up to 64 * CPL pool candidates; knob
// values of a lane's candidates (packed in pairs) are held in registers for
// up to 4 candidates a lane, read from LDS for more.  A round takes the
// largest gain's order bits over the wave (0 marks a candidate already
// picked or absent: every finite gain orders above 0), then the earliest
// candidate that has it: candidate lane + 64 i comes before every candidate
// of a later i, so the first i whose ballot is not empty, and its lowest
// lane, give the winner.  The winners' indices go to win_idx.
template <int CPL>
__device__ void greedy_rounds(const SelectArgs& a, const at_entry* pool, const uint32_t* vals, int have, int m,
                              int* win_idx, int rounds) {
    constexpr int W = MAX_KNOBS / 2;
    const int lane = threadIdx.x & 63;
    const uint32_t all = m >= 32 ? 0xffffffffu : (1u << m) - 1u;
    constexpr bool REG = CPL <= 4;
    constexpr int KR = REG ? CPL : 1;
    float sc[CPL];
    uint32_t fresh[CPL], kv[KR][W];
    uint32_t taken = 0u;   // bit i: candidate lane + 64 i is picked or absent
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
        if (!mine) taken |= 1u << i;
    }
    for (int r = 0; r < rounds; ++r) {
        uint32_t go[CPL], best = 0u;
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            const float g = sc[i] + a.alpha * (float)__popc(fresh[i]);
            const uint32_t o = gain_order(g);
            go[i] = ((taken >> i) & 1u) ? 0u : o;
            best = go[i] > best ? go[i] : best;
        }
        best = wave_max_u32(best);
        int win = -1;
#pragma unroll
        for (int i = 0; i < CPL; ++i) {
            const uint64_t bal = __ballot(go[i] == best);
            if (win < 0 && bal != 0) win = 64 * i + (int)__builtin_ctzll(bal);
        }
        const int wl = win & 63, wi = win >> 6;
        if (wl == lane) taken |= 1u << wi;
        // the knobs whose value the winner adds (its fresh knobs): only
        // candidates with the same value at those knobs lose them
        uint32_t wf = 0u;
#pragma unroll
        for (int i = 0; i < CPL; ++i)
            if (i == wi) wf = fresh[i];
        uint32_t added = (uint32_t)__builtin_amdgcn_readlane((int)wf, wl);
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
        if (lane == 0) win_idx[r] = win;
    }
}

// Four waves per SIMD (the workgroup's sixteen): up to 128 VGPRs, so the
// greedy wave keeps its candidates in registers without spilling.
__global__ __launch_bounds__(SEL_WG) __attribute__((amdgpu_waves_per_eu(1, 4))) void k_select(SelectArgs a) {
    extern __shared__ uint4 sel_lds[];
    uint64_t* key0 = reinterpret_cast<uint64_t*>(sel_lds);                       // [FINAL_MAX]
    uint64_t* key1 = key0 + FINAL_MAX;                                           // [FINAL_MAX]
    uint32_t* bits0 = reinterpret_cast<uint32_t*>(key1 + FINAL_MAX);             // [FINAL_MAX]
    uint32_t* bits1 = bits0 + FINAL_MAX;                                         // [FINAL_MAX]
    at_entry* pool = reinterpret_cast<at_entry*>(bits1 + FINAL_MAX);             // [POOL_MAX]
    uint32_t* vals = reinterpret_cast<uint32_t*>(pool + POOL_MAX);               // [POOL_MAX][MAX_KNOBS / 2]
    uint64_t* picked = reinterpret_cast<uint64_t*>(vals + POOL_MAX * (MAX_KNOBS / 2));   // [PICK_MAX], pick order
    uint64_t* sorted = picked + PICK_MAX;                                        // [PICK_MAX], ascending
    __shared__ int wsum[SEL_WG / 64];
    const int tid = threadIdx.x, lane = tid & 63;
    const SpaceDesc& sd = *a.desc;

    // the pool: the `pool` best distinct candidates
    int nsort = 1;
    while (nsort < a.n) nsort <<= 1;
    const RecBuf v{key0, bits0}, w{key1, bits1};
    load_slice(a.src, 0, a.n, nsort, v);
    const RecBuf sorted_c = merge_sort<FINAL_MAX / SEL_WG>(v, w, nsort, a.run < nsort ? a.run : nsort);
    const int have = compact_distinct(sorted_c, nsort, pool, a.pool, a.pool, wsum);

    // knob values of the pool candidates, packed in pairs (indices fit 32
    // bits: a space has fewer than 2^32 configurations)
    const int m = sd.n_knobs;
    for (int c = tid; c < have; c += SEL_WG) {
        uint32_t cfg = (uint32_t)pool[c].cfg;
        uint32_t kv[MAX_KNOBS];
#pragma unroll
        for (int j = 0; j < MAX_KNOBS; ++j) {
            kv[j] = 0u;
            if (j < m) {
                const uint32_t rdx = (uint32_t)sd.radix[j];
                const uint32_t q = cfg / rdx;
                kv[j] = q;
                cfg -= q * rdx;
            }
        }
#pragma unroll
        for (int j = 0; j < MAX_KNOBS / 2; ++j) vals[c * (MAX_KNOBS / 2) + j] = kv[2 * j] | (kv[2 * j + 1] << 16);
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
        int rank = 0;
        for (int j = 0; j < rounds; ++j) rank += picked[j] < x ? 1 : 0;
        sorted[rank] = x;
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();

    // epsilon-greedy draws, then empty slots
    const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
    int n_sel = rounds, slot = rounds;
    for (int i = 0; i < a.n_random; ++i) {
        const uint64_t remaining = sd.n_configs - (uint64_t)n_sel;
        if (remaining == 0) break;
        const U4 r = philox(k0, k1, U4{(uint32_t)i, 0u, 5u, 0u});
        const uint64_t u = ((uint64_t)r.y << 32) | r.x;
        const uint64_t k = __umul64hi(u, remaining);
        // j = #{positions p with sorted[p] - p <= k}: those picks lie at or
        // below the drawn index, which is then k + j
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
        if (lane == 0) {
            sorted[j] = cfg;
            at_entry e;
            e.cfg = cfg;
            e.score = 0.0f;
            e.flag = 2u;
            a.out[slot] = e;
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_wave_barrier();
        ++n_sel;
        ++slot;
    }
    for (int q = slot + lane; q < a.n_greedy + a.n_random; q += 64) a.out[q] = empty_entry();
}

size_t select_lds_bytes() {
    return (size_t)FINAL_MAX * (8 + 4) * 2 + (size_t)POOL_MAX * sizeof(at_entry) +
           (size_t)POOL_MAX * (MAX_KNOBS / 2) * 4 + (size_t)PICK_MAX * 8 * 2;
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
    int run = 1;
    const at_entry* src = cand;
    int64_t n = n_cand;
    void* bufs[2] = {nullptr, nullptr};
    const int64_t need = select_scratch_entries(n_cand, pool);
    const bool own = need > 0 && !scratch;   // stream-ordered buffers of our own
    if (need > 0 && scratch) {
        if (need > SELECT_SCRATCH_ENTRIES) return hipErrorInvalidValue;
        bufs[0] = scratch;
        bufs[1] = scratch + SELECT_SCRATCH_ENTRIES;
    } else if (own) {
        const size_t bytes = (size_t)need * sizeof(at_entry);
        for (void*& b : bufs) {
            e = hipMallocAsync(&b, bytes, stream);
            if (e != hipSuccess) {
                for (void* x : bufs)
                    if (x) (void)hipFreeAsync(x, stream);
                return e;
            }
        }
    }
    int cur = 0;
    while (n > FINAL_MAX) {
        const int64_t groups = (n + CHUNK - 1) / CHUNK;
        hipLaunchKernelGGL(k_reduce, dim3((unsigned)groups), dim3(SEL_WG), 0, stream, src, n, run, keep, slots,
                           static_cast<at_entry*>(bufs[cur]));
        if ((e = hipGetLastError()) != hipSuccess) break;
        src = static_cast<const at_entry*>(bufs[cur]);
        n = groups * slots;
        run = slots;
        cur ^= 1;
    }
    if (e != hipSuccess) {
        if (own)
            for (void* x : bufs)
                if (x) (void)hipFreeAsync(x, stream);
        return e;
    }
    SelectArgs a{};
    a.desc = static_cast<const SpaceDesc*>(sp.d_descs.p);
    a.src = src;
    a.n = n;
    a.run = run;
    a.pool = pool;
    a.n_greedy = n_greedy;
    a.alpha = alpha;
    a.n_random = n_random;
    a.seed = seed;
    a.out = out;
    hipLaunchKernelGGL(k_select, dim3(1), dim3(SEL_WG), select_lds_bytes(), stream, a);
    e = hipGetLastError();
    if (own)
        for (void* b : bufs)
            if (b) (void)hipFreeAsync(b, stream);
    return e;
}

}  // namespace at
