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
// k_pool_partial: each workgroup sorts a slice of up to SORT_N entries in
// LDS (bitonic), drops repeated indices and writes its `pool` best.
// k_select (one workgroup): merges the partial results the same way, then
// one thread per pool candidate runs the greedy rounds (block-wide arg-max
// of the gains, then every candidate clears the knobs the winner covers),
// and thread 0 draws the random configurations.
#include <mutex>

#include "at_chain.h"

namespace at {
namespace {

using namespace dev;

constexpr int SEL_WG = 1024;
constexpr int SORT_N = 4096;     // entries one workgroup sorts (64 KB of LDS)
constexpr int MERGE_MAX = 4096;  // entries the final workgroup sorts (64 KB)
constexpr int POOL_MAX = SEL_WG; // one thread per pool candidate
constexpr int PICK_MAX = 2048;   // greedy plus random picks

// Sort key: (order of the score, descending; index ascending), invalid
// entries last.  -0.0 counts as +0.0, as in a float comparison.
struct Key {
    uint32_t s;   // larger score -> smaller s
    uint64_t cfg;
};

__device__ __forceinline__ Key key_of(const at_entry& e) {
    Key k;
    if (!e.flag) {
        k.s = 0xffffffffu;
        k.cfg = ~0ull;
        return k;
    }
    uint32_t b = __float_as_uint(e.score);
    if (b == 0x80000000u) b = 0u;
    const uint32_t asc = (b & 0x80000000u) ? ~b : (b | 0x80000000u);   // ascending float order
    k.s = ~asc;
    k.cfg = e.cfg;
    return k;
}

__device__ __forceinline__ bool key_less(const Key& a, const Key& b) {
    return a.s < b.s || (a.s == b.s && a.cfg < b.cfg);
}

// Bitonic sort of n (a power of two) entries in LDS by key; all threads call.
__device__ void bitonic_sort(at_entry* v, int n) {
    for (int size = 2; size <= n; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            __syncthreads();
            for (int i = threadIdx.x; i < n / 2; i += blockDim.x) {
                const int lo = 2 * i - (i & (stride - 1));
                const int hi = lo + stride;
                const bool up = (lo & size) == 0;
                const at_entry a = v[lo], b = v[hi];
                const bool swap = up ? key_less(key_of(b), key_of(a)) : key_less(key_of(a), key_of(b));
                if (swap) {
                    v[lo] = b;
                    v[hi] = a;
                }
            }
        }
    }
    __syncthreads();
}

// Exclusive prefix sum of x over the block's threads (thread order); the
// total goes to *total.  All threads call; uses wsum[SEL_WG / 64].
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

// Sorted entries v[0..n) (n a power of two): the first `keep` distinct valid
// ones (an index equal to its predecessor's is dropped) go to out[0..keep),
// the rest of out is cleared; returns how many were found (at most keep).
// Thread t looks after the consecutive entries [t * per, (t + 1) * per).
// All threads call.
__device__ int compact_distinct(const at_entry* v, int n, at_entry* out, int keep, int* wsum) {
    const int per = n > (int)blockDim.x ? n / (int)blockDim.x : 1;
    const int lo = threadIdx.x * per;
    int cnt = 0;
    for (int i = lo; i < lo + per && i < n; ++i) cnt += (v[i].flag && (i == 0 || v[i].cfg != v[i - 1].cfg)) ? 1 : 0;
    int total = 0;
    int pos = block_exclusive_scan(cnt, wsum, &total);
    for (int i = lo; i < lo + per && i < n; ++i) {
        if (v[i].flag && (i == 0 || v[i].cfg != v[i - 1].cfg)) {
            if (pos < keep) out[pos] = v[i];
            ++pos;
        }
    }
    const int have = total < keep ? total : keep;
    for (int i = have + (int)threadIdx.x; i < keep; i += blockDim.x) {
        at_entry z;
        z.cfg = 0;
        z.score = 0.0f;
        z.flag = 0u;
        out[i] = z;
    }
    __syncthreads();
    return have;
}

__device__ __forceinline__ at_entry empty_entry() {
    at_entry z;
    z.cfg = 0;
    z.score = 0.0f;
    z.flag = 0u;
    return z;
}

// Workgroup b: entries [b * SORT_N, ...) of src -> its `keep` best distinct at dst + b * keep.
__global__ __launch_bounds__(SEL_WG) void k_pool_partial(const at_entry* __restrict__ src, int64_t n, int keep,
                                                          at_entry* __restrict__ dst) {
    __shared__ at_entry v[SORT_N];
    __shared__ int wsum[SEL_WG / 64];
    const int64_t base = (int64_t)blockIdx.x * SORT_N;
    for (int i = threadIdx.x; i < SORT_N; i += blockDim.x) v[i] = base + i < n ? src[base + i] : empty_entry();
    bitonic_sort(v, SORT_N);
    compact_distinct(v, SORT_N, dst + (int64_t)blockIdx.x * keep, keep, wsum);
}

struct SelectArgs {
    const SpaceDesc* desc;
    const at_entry* src;      // sorted input candidates, or partial results
    int64_t n;                // entries in src (at most MERGE_MAX)
    int pool;
    int n_greedy;
    float alpha;
    int n_random;
    uint64_t seed;
    at_entry* out;            // [n_greedy + n_random]
};

__global__ __launch_bounds__(SEL_WG) void k_select(SelectArgs a) {
    extern __shared__ uint4 sel_lds[];
    at_entry* v = reinterpret_cast<at_entry*>(sel_lds);                  // [MERGE_MAX]
    at_entry* pool = v + MERGE_MAX;                                      // [POOL_MAX]
    uint16_t* vals = reinterpret_cast<uint16_t*>(pool + POOL_MAX);       // [POOL_MAX][MAX_KNOBS]
    uint64_t* picked = reinterpret_cast<uint64_t*>(vals + POOL_MAX * MAX_KNOBS);   // [PICK_MAX], ascending
    __shared__ float w_gain[SEL_WG / 64];
    __shared__ int w_idx[SEL_WG / 64];
    __shared__ int s_win;
    __shared__ int wsum[SEL_WG / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const SpaceDesc& sd = *a.desc;

    // the pool: the `pool` best distinct candidates
    int nsort = 1;
    while (nsort < a.n) nsort <<= 1;
    for (int i = tid; i < nsort; i += SEL_WG) v[i] = i < a.n ? a.src[i] : empty_entry();
    bitonic_sort(v, nsort);
    const int have = compact_distinct(v, nsort, pool, a.pool, wsum);

    // knob values of the pool candidates; mask of knobs not yet covered
    const int m = sd.n_knobs;
    uint32_t fresh = 0u;
    float score = 0.0f;
    const bool mine = tid < have;
    if (mine) {
        uint64_t cfg = pool[tid].cfg;
        score = pool[tid].score;
        for (int j = 0; j < m; ++j) {
            const uint64_t q = cfg / sd.radix[j];
            vals[tid * MAX_KNOBS + j] = (uint16_t)q;
            cfg -= q * sd.radix[j];
        }
        fresh = (1u << m) - 1u;
    }
    bool taken = !mine;
    const int rounds = a.n_greedy < have ? a.n_greedy : have;
    __syncthreads();
    for (int r = 0; r < rounds; ++r) {
        // gain of every untaken candidate; block arg-max by (gain, -index)
        float g = -INFINITY;
        int gi = 0x7fffffff;
        if (!taken) {
            const float cov = a.alpha * (float)__popc(fresh);
            g = score + cov;
            gi = tid;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const float og = __shfl_xor(g, off);
            const int oi = __shfl_xor(gi, off);
            if (og > g || (og == g && oi < gi)) {
                g = og;
                gi = oi;
            }
        }
        if (lane == 0) {
            w_gain[wave] = g;
            w_idx[wave] = gi;
        }
        __syncthreads();
        if (tid == 0) {
            float bg = w_gain[0];
            int bi = w_idx[0];
            for (int w = 1; w < SEL_WG / 64; ++w)
                if (w_gain[w] > bg || (w_gain[w] == bg && w_idx[w] < bi)) {
                    bg = w_gain[w];
                    bi = w_idx[w];
                }
            s_win = bi;
            at_entry e;
            e.cfg = pool[bi].cfg;
            e.score = pool[bi].score;
            e.flag = 1u;
            a.out[r] = e;
            picked[r] = e.cfg;
        }
        __syncthreads();
        const int win = s_win;
        if (tid == win) taken = true;
        if (mine) {
            for (int j = 0; j < m; ++j)
                if (vals[tid * MAX_KNOBS + j] == vals[win * MAX_KNOBS + j]) fresh &= ~(1u << j);
        }
        __syncthreads();
    }

    // epsilon-greedy, then empty slots
    if (tid == 0) {
        int n_sel = rounds;
        // ascending order of the greedy picks (insertion sort)
        for (int i = 1; i < n_sel; ++i) {
            const uint64_t x = picked[i];
            int j = i - 1;
            while (j >= 0 && picked[j] > x) {
                picked[j + 1] = picked[j];
                --j;
            }
            picked[j + 1] = x;
        }
        const uint32_t k0 = (uint32_t)a.seed, k1 = (uint32_t)(a.seed >> 32);
        int slot = rounds;
        for (int i = 0; i < a.n_random; ++i) {
            const uint64_t remaining = sd.n_configs - (uint64_t)n_sel;
            if (remaining == 0) break;
            const U4 r = philox(k0, k1, U4{(uint32_t)i, 0u, 5u, 0u});
            const uint64_t u = ((uint64_t)r.y << 32) | r.x;
            uint64_t cfg = __umul64hi(u, remaining);
            int pos = 0;
            while (pos < n_sel && picked[pos] <= cfg) {
                ++cfg;
                ++pos;
            }
            for (int j = n_sel; j > pos; --j) picked[j] = picked[j - 1];
            picked[pos] = cfg;
            ++n_sel;
            at_entry e;
            e.cfg = cfg;
            e.score = 0.0f;
            e.flag = 2u;
            a.out[slot++] = e;
        }
        for (; slot < a.n_greedy + a.n_random; ++slot) a.out[slot] = empty_entry();
    }
}

size_t select_lds_bytes() {
    return (size_t)MERGE_MAX * sizeof(at_entry) + (size_t)POOL_MAX * sizeof(at_entry) +
           (size_t)POOL_MAX * MAX_KNOBS * 2 + (size_t)PICK_MAX * 8;
}

}  // namespace

int select_pool_max() { return POOL_MAX; }
int select_pick_max() { return PICK_MAX; }

// Entries of each of the two partial-result buffers the reduction of n_cand
// candidates needs (0 when n_cand fits the final workgroup).
int64_t select_scratch_entries(int64_t n_cand, int pool) {
    if (n_cand <= MERGE_MAX) return 0;
    const int keep = pool > 0 ? pool : 1;
    return (n_cand + SORT_N - 1) / SORT_N * keep;
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
    // reduce the candidates to at most MERGE_MAX entries: each level keeps
    // the `keep` best distinct of every SORT_N-entry slice (a quarter or less)
    const int keep = pool > 0 ? pool : 1;
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
    while (n > MERGE_MAX) {
        const int64_t groups = (n + SORT_N - 1) / SORT_N;
        hipLaunchKernelGGL(k_pool_partial, dim3((unsigned)groups), dim3(SEL_WG), 0, stream, src, n, keep,
                           static_cast<at_entry*>(bufs[cur]));
        if ((e = hipGetLastError()) != hipSuccess) break;
        src = static_cast<const at_entry*>(bufs[cur]);
        n = groups * keep;
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
