// C ABI of the autotensor library: handle lifetimes, argument checks, status
// codes and the host-side threshold helper.  Every compute entry point
// validates its arguments and then enqueues HIP kernels on the caller's
// stream.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>

#include "at_internal.h"

namespace at {

namespace {
thread_local std::string g_last_error;

// Bytes one workgroup of the chain-local path may stream per step for the
// path to be chosen by default.  Measured on MI355X: the chain-local path
// wins with its ensemble resident in LDS (GEMM 512^3: 2.5 ms against 6.4 ms
// per run) and streaming about 0.4 MB per step (conv2d C2: 5.7 against
// 9.2 ms), and loses at 1.5 MB per step (twelve conv2d workloads: 33 against
// 20 ms).
constexpr double LOCAL_AUTO_BYTES = 768.0 * 1024;

template <class T>
at_status upload(DeviceBuf& buf, const T* host, size_t count) {
    buf.bytes = count * sizeof(T);
    if (buf.bytes == 0) buf.bytes = 16;
    hipError_t e = hipMalloc(&buf.p, buf.bytes);
    if (e != hipSuccess) {
        buf.p = nullptr;
        return hip_fail(e, "hipMalloc");
    }
    if (count) {
        e = hipMemcpy(buf.p, host, count * sizeof(T), hipMemcpyHostToDevice);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
    }
    return AT_OK;
}

at_status alloc_zero(DeviceBuf& buf, size_t bytes) {
    buf.bytes = bytes ? bytes : 16;
    hipError_t e = hipMalloc(&buf.p, buf.bytes);
    if (e != hipSuccess) {
        buf.p = nullptr;
        return hip_fail(e, "hipMalloc");
    }
    e = hipMemset(buf.p, 0, buf.bytes);
    if (e != hipSuccess) return hip_fail(e, "hipMemset");
    return AT_OK;
}

// Largest single space whose configurations are all scanned for constant
// loop-context features (a few milliseconds of one GPU at this size).
constexpr uint64_t FEATURE_SCAN_MAX = (uint64_t)1 << 28;

void release(DeviceBuf& buf);

// Constant loop-context features of a single space (see at_space_s).
at_status scan_constant_features(at_space_s& sp) {
    const SpaceDesc& d = sp.descs[0];
    sp.fconst.clear();
    if (d.n_configs > FEATURE_SCAN_MAX) return AT_OK;
    const int F = d.n_features;
    DeviceBuf buf;
    at_status st = alloc_zero(buf, (size_t)2 * F * 4);
    if (st != AT_OK) return st;
    uint32_t* flags = static_cast<uint32_t*>(buf.p);
    hipError_t e = launch_feature_scan(sp, flags, flags + F, nullptr);
    std::vector<uint32_t> host((size_t)2 * F);
    if (e == hipSuccess) e = hipMemcpy(host.data(), buf.p, host.size() * 4, hipMemcpyDeviceToHost);
    release(buf);
    if (e != hipSuccess) return hip_fail(e, "feature scan");
    sp.fconst.resize(F);
    // a constant above the annealing features' range stays in the tile (the
    // walk's threshold compare is exact only within that range)
    for (int f = 0; f < F; ++f)
        sp.fconst[f] = (host[f] != 0u || host[F + f] > SA_FEATURE_MAX) ? 0xff : (uint8_t)host[F + f];
    return AT_OK;
}

// Tile layout of the tree-partitioned path (see at_space_s): the varying
// features only, in feature order, when that halves the tile slot (a power
// of two of at least 256 bytes per wave: more waves or trees fit in LDS);
// otherwise every feature in order.
at_status build_feature_tables(at_space_s& sp) {
    const int F = sp.descs[0].n_features, Q = (F + 3) / 4;
    int nvar = 0;
    for (uint8_t v : sp.fconst) nvar += v == 0xff;
    const int qc = nvar > 0 ? (nvar + 3) / 4 : 1;
    auto slot = [](int q) {
        int s = 256;
        while (s < q * 256) s <<= 1;
        return s;
    };
    const bool compact = !sp.fconst.empty() && slot(qc) < slot(Q);
    sp.tile_q = compact ? qc : Q;
    std::vector<uint16_t> map(256, 0);
    std::vector<uint8_t> src((size_t)4 * sp.tile_q, 0xff);
    for (int f = 0, p = 0; f < F; ++f) {
        if (compact && sp.fconst[f] != 0xff) {
            map[f] = (uint16_t)(0x100 | sp.fconst[f]);
        } else {
            map[f] = (uint16_t)p;
            src[p++] = (uint8_t)f;
        }
    }
    at_status st = upload(sp.d_fmap, map.data(), map.size());
    if (st == AT_OK) st = upload(sp.d_fsrc, src.data(), src.size());
    return st;
}

// LDS images of a space's members and, for a set, the image of each block
// of STAGE_CHAINS chains (see at_space_s).
at_status build_stage(at_space_s& sp) {
    std::vector<int> fits(sp.n_spaces, 0);
    size_t need = 0;
    for (int i = 0; i < sp.n_spaces; ++i) {
        const size_t nf = sp.host_factors[i].size();
        fits[i] = nf <= (size_t)STAGE_FAC_MAX;
        if (fits[i]) need = std::max(need, (size_t)STAGE_DESC_BYTES + nf * 8);
    }
    const size_t stride = (need + STAGE_ALIGN - 1) / STAGE_ALIGN * STAGE_ALIGN;
    std::vector<uint8_t> img(stride * sp.n_spaces, 0);
    for (int i = 0; i < sp.n_spaces && stride; ++i) {
        if (!fits[i]) continue;
        SpaceDesc d = sp.descs[i];
        const int32_t base = d.split_off[0];
        for (int a = 0; a < d.n_axes; ++a) d.split_off[a] -= base;
        uint8_t* dst = img.data() + stride * i;
        std::memcpy(dst, &d, sizeof d);
        std::memcpy(dst + STAGE_DESC_BYTES, sp.host_factors[i].data(), sp.host_factors[i].size() * 8);
    }
    sp.stage_stride = (int)stride;
    at_status st = upload(sp.d_stage, img.data(), img.size());
    if (st != AT_OK) return st;
    if (sp.n_spaces == 1) {
        sp.stage_single = fits[0] ? 0 : -1;
        return AT_OK;
    }
    const int64_t n = sp.chain_offsets.back();
    const int64_t blocks = (n + STAGE_CHAINS - 1) / STAGE_CHAINS;
    std::vector<int32_t> ws((size_t)blocks, -1);
    int w = 0;
    for (int64_t b = 0; b < blocks; ++b) {
        const int64_t lo = b * STAGE_CHAINS, hi = std::min(n, lo + STAGE_CHAINS) - 1;
        while (w + 1 < sp.n_spaces && sp.chain_offsets[w + 1] <= lo) ++w;
        int wh = w;
        while (wh + 1 < sp.n_spaces && sp.chain_offsets[wh + 1] <= hi) ++wh;
        ws[(size_t)b] = (wh == w && fits[w]) ? w : -1;
    }
    return upload(sp.d_wg_space, ws.data(), ws.size());
}

void release(DeviceBuf& buf) {
    if (buf.p) (void)hipFree(buf.p);
    buf.p = nullptr;
    buf.bytes = 0;
}

int current_device() {
    int d = 0;
    (void)hipGetDevice(&d);
    return d;
}

// Makes the handle's device current for the duration of a call.
struct DeviceGuard {
    int prev = 0;
    bool switched = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
            switched = hipSetDevice(dev) == hipSuccess;
        }
    }
    ~DeviceGuard() {
        if (switched) (void)hipSetDevice(prev);
    }
};

at_status finish_launch(hipError_t e, const char* what) {
    if (e != hipSuccess) return hip_fail(e, what);
    return AT_OK;
}

}  // namespace

at_status fail(at_status st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

at_status hip_fail(hipError_t e, const char* what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return e == hipErrorOutOfMemory ? AT_E_OOM : AT_E_HIP;
}

}  // namespace at

using namespace at;

extern "C" {

const char* at_last_error(void) { return g_last_error.c_str(); }

at_status at_space_create(int tmpl, const int64_t* shape, int nshape, at_space_t* out) {
    if (!out) return fail(AT_E_INVALID, "at_space_create: out is NULL");
    *out = nullptr;
    SpaceDesc d;
    std::vector<uint64_t> factors;
    at_status st = build_space(tmpl, shape, nshape, d, factors);
    if (st != AT_OK) return st;
    at_space_s* sp = new (std::nothrow) at_space_s();
    if (!sp) return fail(AT_E_OOM, "at_space_create: host allocation");
    sp->device = current_device();
    sp->tmpl = d.tmpl;
    sp->api_tmpl = tmpl;
    sp->n_spaces = 1;
    sp->descs.push_back(d);
    sp->chain_offsets = {0, 0};
    sp->host_factors.push_back(factors);
    int64_t offs[2] = {0, INT64_MAX};
    if ((st = upload(sp->d_descs, &d, 1)) != AT_OK || (st = upload(sp->d_factors, factors.data(), factors.size())) != AT_OK ||
        (st = upload(sp->d_offsets, offs, 2)) != AT_OK || (st = alloc_zero(sp->d_errors, 8)) != AT_OK ||
        (st = build_stage(*sp)) != AT_OK || (st = scan_constant_features(*sp)) != AT_OK ||
        (st = build_feature_tables(*sp)) != AT_OK) {
        at_space_destroy(sp);
        return st;
    }
    *out = sp;
    return AT_OK;
}

at_status at_space_info(at_space_t space, int* n_knobs, int32_t* knob_sizes, int* n_loops, int* n_features,
                        uint64_t* n_configs) {
    if (!space) return fail(AT_E_INVALID, "at_space_info: NULL space");
    const SpaceDesc& d = space->descs[0];
    if (n_knobs) *n_knobs = d.n_knobs;
    if (knob_sizes)
        for (int j = 0; j < d.n_knobs; ++j) knob_sizes[j] = (int32_t)d.knob_size[j];
    if (n_loops) *n_loops = d.tmpl == AT_TMPL_GEMM ? 10 : 16;
    if (n_features) *n_features = d.n_features;
    if (n_configs) {
        uint64_t total = 0;
        for (const SpaceDesc& x : space->descs) total += x.n_configs;
        *n_configs = space->n_spaces == 1 ? d.n_configs : total;
    }
    return AT_OK;
}

at_status at_spaceset_create(const at_space_t* spaces, int n, const int64_t* chain_offsets, at_space_t* out) {
    if (!out) return fail(AT_E_INVALID, "at_spaceset_create: out is NULL");
    *out = nullptr;
    if (!spaces || !chain_offsets || n < 1) return fail(AT_E_INVALID, "at_spaceset_create: bad arguments");
    if (chain_offsets[0] != 0) return fail(AT_E_INVALID, "at_spaceset_create: chain_offsets[0] must be 0");
    for (int i = 0; i < n; ++i) {
        if (!spaces[i] || spaces[i]->n_spaces != 1) return fail(AT_E_INVALID, "at_spaceset_create: member must be a single space");
        if (chain_offsets[i + 1] < chain_offsets[i]) return fail(AT_E_INVALID, "at_spaceset_create: offsets must ascend");
        if (spaces[i]->api_tmpl != spaces[0]->api_tmpl) return fail(AT_E_MISMATCH, "at_spaceset_create: templates differ");
    }
    at_space_s* sp = new (std::nothrow) at_space_s();
    if (!sp) return fail(AT_E_OOM, "at_spaceset_create: host allocation");
    sp->device = current_device();
    sp->tmpl = spaces[0]->tmpl;
    sp->api_tmpl = spaces[0]->api_tmpl;
    sp->n_spaces = n;
    std::vector<uint64_t> all;
    for (int i = 0; i < n; ++i) {
        SpaceDesc d = spaces[i]->descs[0];
        const int32_t shift = (int32_t)all.size();
        for (int a = 0; a < d.n_axes; ++a) d.split_off[a] += shift;
        const std::vector<uint64_t>& f = spaces[i]->host_factors[0];
        all.insert(all.end(), f.begin(), f.end());
        sp->descs.push_back(d);
        sp->host_factors.push_back(f);
    }
    sp->chain_offsets.assign(chain_offsets, chain_offsets + n + 1);
    // a feature is constant over the set when every member gives it the same
    // value
    sp->fconst = spaces[0]->fconst;
    for (int i = 1; i < n && !sp->fconst.empty(); ++i) {
        const std::vector<uint8_t>& m = spaces[i]->fconst;
        if (m.size() != sp->fconst.size()) {
            sp->fconst.clear();
            break;
        }
        for (size_t f = 0; f < m.size(); ++f)
            if (m[f] != sp->fconst[f]) sp->fconst[f] = 0xff;
    }
    at_status st;
    if ((st = upload(sp->d_descs, sp->descs.data(), sp->descs.size())) != AT_OK ||
        (st = upload(sp->d_factors, all.data(), all.size())) != AT_OK ||
        (st = upload(sp->d_offsets, sp->chain_offsets.data(), sp->chain_offsets.size())) != AT_OK ||
        (st = alloc_zero(sp->d_errors, 8)) != AT_OK || (st = build_stage(*sp)) != AT_OK ||
        (st = build_feature_tables(*sp)) != AT_OK) {
        at_space_destroy(sp);
        return st;
    }
    *out = sp;
    return AT_OK;
}

void at_space_destroy(at_space_t space) {
    if (!space) return;
    DeviceGuard g(space->device);
    release(space->d_descs);
    release(space->d_factors);
    release(space->d_offsets);
    release(space->d_errors);
    release(space->d_stage);
    release(space->d_wg_space);
    release(space->d_fsrc);
    release(space->d_fmap);
    delete space;
}

at_status at_extract_features(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats, at_stream_t stream) {
    if (!space) return fail(AT_E_INVALID, "at_extract_features: NULL space");
    if (space->n_spaces != 1) return fail(AT_E_INVALID, "at_extract_features: takes a single space, not a set");
    if (n < 0) return fail(AT_E_INVALID, "at_extract_features: n < 0");
    if (n == 0) return AT_OK;
    if (!cfgs || !feats) return fail(AT_E_INVALID, "at_extract_features: NULL buffer");
    if (n > ((int64_t)1 << 36)) return fail(AT_E_UNSUPPORTED, "at_extract_features: n too large for one call");
    DeviceGuard g(space->device);
    return finish_launch(launch_extract(*space, cfgs, n, feats, (hipStream_t)stream), "at_extract_features");
}

at_status at_extract_features_full(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                   at_stream_t stream) {
    if (!space) return fail(AT_E_INVALID, "at_extract_features_full: NULL space");
    if (space->n_spaces != 1) return fail(AT_E_INVALID, "at_extract_features_full: takes a single space, not a set");
    if (n < 0) return fail(AT_E_INVALID, "at_extract_features_full: n < 0");
    if (n == 0) return AT_OK;
    if (!cfgs || !feats) return fail(AT_E_INVALID, "at_extract_features_full: NULL buffer");
    if (n > ((int64_t)1 << 36)) return fail(AT_E_UNSUPPORTED, "at_extract_features_full: n too large for one call");
    DeviceGuard g(space->device);
    return finish_launch(launch_extract_full(*space, cfgs, n, feats, (hipStream_t)stream), "at_extract_features_full");
}

at_status at_extract_features_onehot(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                     at_stream_t stream) {
    if (!space) return fail(AT_E_INVALID, "at_extract_features_onehot: NULL space");
    if (space->n_spaces != 1) return fail(AT_E_INVALID, "at_extract_features_onehot: takes a single space, not a set");
    if (n < 0) return fail(AT_E_INVALID, "at_extract_features_onehot: n < 0");
    if (n == 0) return AT_OK;
    if (!cfgs || !feats) return fail(AT_E_INVALID, "at_extract_features_onehot: NULL buffer");
    if (n > ((int64_t)1 << 40)) return fail(AT_E_UNSUPPORTED, "at_extract_features_onehot: n too large");
    DeviceGuard g(space->device);
    return finish_launch(launch_extract_onehot(*space, cfgs, n, feats, (hipStream_t)stream),
                         "at_extract_features_onehot");
}

at_status at_extract_relation_features(at_space_t space, const uint64_t* cfgs, int64_t n, int32_t* feats,
                                       at_stream_t stream) {
    if (!space) return fail(AT_E_INVALID, "at_extract_relation_features: NULL space");
    if (space->n_spaces != 1) return fail(AT_E_INVALID, "at_extract_relation_features: takes a single space, not a set");
    if (n < 0) return fail(AT_E_INVALID, "at_extract_relation_features: n < 0");
    if (n == 0) return AT_OK;
    if (!cfgs || !feats) return fail(AT_E_INVALID, "at_extract_relation_features: NULL buffer");
    if ((reinterpret_cast<uintptr_t>(feats) & 15u) != 0)
        return fail(AT_E_INVALID, "at_extract_relation_features: feats must be 16-byte aligned");
    if (n > ((int64_t)1 << 36)) return fail(AT_E_UNSUPPORTED, "at_extract_relation_features: n too large for one call");
    DeviceGuard g(space->device);
    return finish_launch(launch_relation(*space, cfgs, n, feats, (hipStream_t)stream), "at_extract_relation_features");
}

at_status at_space_errors(at_space_t space, uint64_t* n_out_of_range) {
    if (!space || !n_out_of_range) return fail(AT_E_INVALID, "at_space_errors: NULL argument");
    DeviceGuard g(space->device);
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    uint64_t v = 0;
    e = hipMemcpy(&v, space->d_errors.p, 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy");
    e = hipMemset(space->d_errors.p, 0, 8);
    if (e != hipSuccess) return hip_fail(e, "hipMemset");
    *n_out_of_range = v;
    return AT_OK;
}

at_status at_ensemble_create(int n_trees, int depth, int n_features, const uint8_t* fid, const uint8_t* thr,
                             const float* leaf, at_ensemble_t* out) {
    if (!out) return fail(AT_E_INVALID, "at_ensemble_create: out is NULL");
    *out = nullptr;
    if (!fid || !thr || !leaf) return fail(AT_E_INVALID, "at_ensemble_create: NULL table");
    if (n_trees < 1 || n_trees > 65535) return fail(AT_E_INVALID, "at_ensemble_create: n_trees out of [1, 65535]");
    if (depth < 1 || depth > 12) return fail(AT_E_UNSUPPORTED, "at_ensemble_create: depth out of [1, 12]");
    if (n_features < 1 || n_features > 256) return fail(AT_E_UNSUPPORTED, "at_ensemble_create: n_features out of [1, 256]");
    const size_t n_int = ((size_t)1 << depth) - 1, n_leaf = (size_t)1 << depth, W = (size_t)2 << depth;
    std::vector<uint32_t> words;
    // padded to whole 32 KB blocks so that chunked prefetches stay in bounds
    const size_t padded = ((size_t)n_trees * W + ENSEMBLE_PAD_WORDS - 1) / ENSEMBLE_PAD_WORDS * ENSEMBLE_PAD_WORDS;
    try {
        words.assign(padded, 0u);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    }
    for (size_t t = 0; t < (size_t)n_trees; ++t) {
        uint32_t* tw = words.data() + t * W;
        for (size_t n = 0; n < n_int; ++n) {
            const uint8_t f = fid[t * n_int + n];
            if (f >= n_features) return fail(AT_E_INVALID, "at_ensemble_create: split feature >= n_features");
            // heap node n (0-based) is word n + 1
            tw[n + 1] = ((uint32_t)thr[t * n_int + n] << 16) | tile_offset(f);
        }
        for (size_t j = 0; j < n_leaf; ++j) {
            uint32_t bits;
            std::memcpy(&bits, &leaf[t * n_leaf + j], 4);
            tw[n_leaf + j] = bits;
        }
    }
    // compact form for the annealing kernels (layout in at_internal.h)
    const size_t NB = n_leaf / 2, W16 = NB + n_leaf;
    std::vector<uint32_t> words16;
    try {
        words16.assign((size_t)n_trees * W16, 0u);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    }
    for (size_t t = 0; t < (size_t)n_trees; ++t) {
        uint32_t* tw = words16.data() + t * W16;
        // heap node m (1-based) is node m - 1 of the caller's tables
        auto node = [&](size_t m) { return node16(fid[t * n_int + m - 1], thr[t * n_int + m - 1]); };
        tw[0] = node(1);
        for (size_t p = 1; p < NB; ++p) tw[p] = node(2 * p) | (node(2 * p + 1) << 16);
        std::memcpy(tw + NB, &leaf[t * n_leaf], n_leaf * 4);
    }
    // pointer form for the tree-partitioned annealing path (layout in at_internal.h)
    const size_t W32 = 4 * NB;
    std::vector<uint32_t> words32;
    try {
        words32.assign((size_t)n_trees * W32, 0u);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    }
    for (size_t t = 0; t < (size_t)n_trees; ++t) {
        uint32_t* tw = words32.data() + t * W32;
        auto node = [&](size_t m) {
            const uint32_t rel = m < NB ? (uint32_t)(2 * m) : (uint32_t)(2 * (m - NB));
            return node16(fid[t * n_int + m - 1], thr[t * n_int + m - 1]) | (rel << 16);
        };
        tw[0] = node(1);
        for (size_t p = 1; p < NB; ++p) {
            tw[2 * p] = node(2 * p);
            tw[2 * p + 1] = node(2 * p + 1);
        }
        std::memcpy(tw + 2 * NB, &leaf[t * n_leaf], n_leaf * 4);
    }
    // local forms for the chain-local annealing path (layout in at_internal.h)
    const size_t ts_full = (size_t)local_tree_stride((int)W16), ts_nodes = (size_t)local_tree_stride((int)NB);
    std::vector<uint32_t> local_full, local_nodes;
    try {
        local_full.assign((size_t)n_trees * ts_full + 4, 0u);
        local_nodes.assign((size_t)n_trees * ts_nodes + 4, 0u);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    }
    for (size_t t = 0; t < (size_t)n_trees; ++t) {
        std::memcpy(local_full.data() + t * ts_full, words16.data() + t * W16, W16 * 4);
        std::memcpy(local_nodes.data() + t * ts_nodes, words16.data() + t * W16, NB * 4);
    }
    // split form: tops (levels 0 .. d-2) and last-level records
    const size_t top_words = depth >= 2 ? NB / 2 : 1;
    const size_t ts_top = (size_t)local_tree_stride((int)top_words);
    std::vector<uint32_t> local_top;
    std::vector<uint32_t> tail;
    try {
        local_top.assign((size_t)n_trees * ts_top + 4, 0u);
        tail.assign((size_t)n_trees * NB * 4, 0u);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    }
    for (size_t t = 0; t < (size_t)n_trees && depth >= 2; ++t) {
        std::memcpy(local_top.data() + t * ts_top, words16.data() + t * W16, top_words * 4);
        for (size_t j = 0; j < NB; ++j) {
            // last-level node m = 2^(d-1) + j (1-based heap); leaves 2m, 2m+1
            const size_t m = NB + j;
            uint32_t* r = tail.data() + (t * NB + j) * 4;
            r[0] = node16(fid[t * n_int + m - 1], thr[t * n_int + m - 1]);
            std::memcpy(&r[1], &leaf[t * n_leaf + 2 * m - n_leaf], 4);
            std::memcpy(&r[2], &leaf[t * n_leaf + 2 * m + 1 - n_leaf], 4);
        }
    }
    at_ensemble_s* e = new (std::nothrow) at_ensemble_s();
    if (!e) return fail(AT_E_OOM, "at_ensemble_create: host allocation");
    e->device = current_device();
    at_status st = upload(e->d_words, words.data(), words.size());
    if (st == AT_OK) st = upload(e->d_words16, words16.data(), words16.size());
    if (st == AT_OK) st = upload(e->d_words32, words32.data(), words32.size());
    if (st == AT_OK) st = upload(e->d_local_full, local_full.data(), local_full.size());
    if (st == AT_OK) st = upload(e->d_local_nodes, local_nodes.data(), local_nodes.size());
    if (st == AT_OK) st = upload(e->d_local_top, local_top.data(), local_top.size());
    if (st == AT_OK) st = upload(e->d_tail, tail.data(), tail.size());
    if (st != AT_OK) {
        at_ensemble_destroy(e);
        return st;
    }
    e->desc.n_trees = n_trees;
    e->desc.depth = depth;
    e->desc.n_features = n_features;
    e->desc.words_per_tree = (int32_t)W;
    e->desc.words = static_cast<const uint32_t*>(e->d_words.p);
    e->desc.words16 = static_cast<const uint32_t*>(e->d_words16.p);
    e->desc.words32 = static_cast<const uint32_t*>(e->d_words32.p);
    e->desc.local_full = static_cast<const uint32_t*>(e->d_local_full.p);
    e->desc.local_nodes = static_cast<const uint32_t*>(e->d_local_nodes.p);
    e->desc.local_top = static_cast<const uint32_t*>(e->d_local_top.p);
    e->desc.tail = static_cast<const uint4*>(e->d_tail.p);
    *out = e;
    return AT_OK;
}

// ---------------------------------------------------------------------------
// Trained trees of any shape: node lists padded to full heap trees.  A leaf
// above the last level becomes a split that always goes left (feature 0,
// threshold 255, while features stay below 255) over two subtrees that both
// end in copies of the leaf, so every row still reaches the leaf's value.
// Float thresholds become integers: for an integer x, x < t holds exactly
// when x < ceil(t).
// ---------------------------------------------------------------------------
namespace {

// Checks the lists of tree t (a binary tree rooted at its first node: every
// child in range, each node reached once) and returns its deepest leaf's
// level in *depth.
at_status tree_shape(int t, const int32_t* offsets, const int32_t* left, const int32_t* right, int* depth) {
    const int64_t base = offsets[t], m = (int64_t)offsets[t + 1] - offsets[t];
    if (base < 0 || m < 1) return fail(AT_E_INVALID, "trees: tree " + std::to_string(t) + " has no nodes");
    std::vector<uint8_t> seen((size_t)m, 0);
    std::vector<std::pair<int32_t, int>> stack{{0, 0}};
    int deepest = 0;
    seen[0] = 1;
    while (!stack.empty()) {
        const auto [i, lev] = stack.back();
        stack.pop_back();
        const int32_t l = left[base + i], r = right[base + i];
        if (l < 0) {
            deepest = lev > deepest ? lev : deepest;
            continue;
        }
        for (const int32_t ch : {l, r}) {
            if (ch < 0 || ch >= m || seen[ch])
                return fail(AT_E_INVALID, "trees: tree " + std::to_string(t) + " node " + std::to_string(i) +
                                              " has a child out of range or reached twice");
            seen[ch] = 1;
            stack.push_back({ch, lev + 1});
        }
    }
    *depth = deepest;
    return AT_OK;
}

uint8_t int_threshold(float t) {
    if (!(t > 0.0f)) return 0;              // x < t never holds for x >= 0
    if (t > 255.0f) return 255;
    return (uint8_t)std::ceil(t);
}

// Heap node h of a depth-D tree from list node i of tree t at level lev.
void pad_node(const int32_t* left, const int32_t* right, const int32_t* feature, const float* threshold,
              const float* value, int64_t base, int32_t i, size_t h, int lev, int D, uint8_t* fid, uint8_t* thr,
              float* leaf) {
    const size_t n_int = ((size_t)1 << D) - 1;
    if (lev == D) {
        leaf[h - n_int] = value[base + i];
        return;
    }
    const bool split = left[base + i] >= 0;
    fid[h] = split ? (uint8_t)feature[base + i] : 0;
    thr[h] = split ? int_threshold(threshold[base + i]) : 255;
    pad_node(left, right, feature, threshold, value, base, split ? left[base + i] : i, 2 * h + 1, lev + 1, D, fid,
             thr, leaf);
    pad_node(left, right, feature, threshold, value, base, split ? right[base + i] : i, 2 * h + 2, lev + 1, D, fid,
             thr, leaf);
}

}  // namespace

at_status at_trees_depth(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                         int* depth) {
    if (!depth) return fail(AT_E_INVALID, "at_trees_depth: depth is NULL");
    *depth = -1;
    if (n_trees < 1 || n_trees > 65535) return fail(AT_E_INVALID, "at_trees_depth: n_trees out of [1, 65535]");
    if (!tree_offsets || !left || !right) return fail(AT_E_INVALID, "at_trees_depth: NULL list");
    int deepest = 0;
    for (int t = 0; t < n_trees; ++t) {
        int d = 0;
        const at_status st = tree_shape(t, tree_offsets, left, right, &d);
        if (st != AT_OK) return st;
        deepest = d > deepest ? d : deepest;
    }
    *depth = deepest;
    return AT_OK;
}

at_status at_trees_pad(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                       const int32_t* feature, const float* threshold, const float* value, int n_features, int depth,
                       uint8_t* fid, uint8_t* thr, float* leaf) {
    if (!feature || !threshold || !value || !fid || !thr || !leaf)
        return fail(AT_E_INVALID, "at_trees_pad: NULL array");
    if (n_features < 1 || n_features > 256) return fail(AT_E_UNSUPPORTED, "at_trees_pad: n_features out of [1, 256]");
    if (depth < 1 || depth > 12) return fail(AT_E_UNSUPPORTED, "at_trees_pad: depth out of [1, 12]");
    int need = 0;
    at_status st = at_trees_depth(n_trees, tree_offsets, left, right, &need);
    if (st != AT_OK) return st;
    if (need > depth) return fail(AT_E_INVALID, "at_trees_pad: a leaf lies below the requested depth");
    for (int t = 0; t < n_trees; ++t)
        for (int64_t j = tree_offsets[t]; j < tree_offsets[t + 1]; ++j) {
            if (left[j] < 0) continue;
            if (feature[j] < 0 || feature[j] >= n_features)
                return fail(AT_E_INVALID, "at_trees_pad: split feature out of [0, n_features)");
            if (std::isnan(threshold[j])) return fail(AT_E_INVALID, "at_trees_pad: NaN threshold");
        }
    const size_t n_int = ((size_t)1 << depth) - 1, n_leaf = (size_t)1 << depth;
    for (int t = 0; t < n_trees; ++t)
        pad_node(left, right, feature, threshold, value, tree_offsets[t], 0, 0, 0, depth, fid + t * n_int,
                 thr + t * n_int, leaf + t * n_leaf);
    return AT_OK;
}

at_status at_ensemble_import(int n_trees, const int32_t* tree_offsets, const int32_t* left, const int32_t* right,
                             const int32_t* feature, const float* threshold, const float* value, int n_features,
                             at_ensemble_t* out) {
    if (!out) return fail(AT_E_INVALID, "at_ensemble_import: out is NULL");
    *out = nullptr;
    int depth = 0;
    at_status st = at_trees_depth(n_trees, tree_offsets, left, right, &depth);
    if (st != AT_OK) return st;
    depth = depth < 1 ? 1 : depth;
    if (depth > 12) return fail(AT_E_UNSUPPORTED, "at_ensemble_import: a leaf lies deeper than level 12");
    const size_t n_int = ((size_t)1 << depth) - 1, n_leaf = (size_t)1 << depth;
    std::vector<uint8_t> fid, thr;
    std::vector<float> leaf;
    try {
        fid.assign((size_t)n_trees * n_int, 0);
        thr.assign((size_t)n_trees * n_int, 0);
        leaf.assign((size_t)n_trees * n_leaf, 0.0f);
    } catch (...) {
        return fail(AT_E_OOM, "at_ensemble_import: host allocation");
    }
    st = at_trees_pad(n_trees, tree_offsets, left, right, feature, threshold, value, n_features, depth, fid.data(),
                      thr.data(), leaf.data());
    if (st != AT_OK) return st;
    return at_ensemble_create(n_trees, depth, n_features, fid.data(), thr.data(), leaf.data(), out);
}

void at_ensemble_destroy(at_ensemble_t ens) {
    if (!ens) return;
    DeviceGuard g(ens->device);
    release(ens->d_words);
    release(ens->d_words16);
    release(ens->d_words32);
    release(ens->d_local_full);
    release(ens->d_local_nodes);
    release(ens->d_local_top);
    release(ens->d_tail);
    delete ens;
}

at_status at_gbt_predict(at_ensemble_t ens, const int32_t* feats, int64_t n, float* scores, uint16_t* leaves,
                         at_stream_t stream) {
    if (!ens) return fail(AT_E_INVALID, "at_gbt_predict: NULL ensemble");
    if (n < 0) return fail(AT_E_INVALID, "at_gbt_predict: n < 0");
    if (n == 0) return AT_OK;
    if (!feats || !scores) return fail(AT_E_INVALID, "at_gbt_predict: NULL buffer");
    if (n > ((int64_t)1 << 40)) return fail(AT_E_UNSUPPORTED, "at_gbt_predict: n too large");
    DeviceGuard g(ens->device);
    return finish_launch(launch_predict(ens->desc, feats, n, scores, leaves, false, (hipStream_t)stream),
                         "at_gbt_predict");
}

at_status at_gbt_predict_global_local(at_ensemble_t global, const int32_t* feats_global, at_ensemble_t local,
                                      const int32_t* feats_local, int64_t n, float* scores, at_stream_t stream) {
    if (!global || !local) return fail(AT_E_INVALID, "at_gbt_predict_global_local: NULL ensemble");
    if (global->device != local->device) return fail(AT_E_INVALID, "at_gbt_predict_global_local: ensembles on different devices");
    if (n < 0) return fail(AT_E_INVALID, "at_gbt_predict_global_local: n < 0");
    if (n == 0) return AT_OK;
    if (!feats_global || !feats_local || !scores) return fail(AT_E_INVALID, "at_gbt_predict_global_local: NULL buffer");
    if (n > ((int64_t)1 << 40)) return fail(AT_E_UNSUPPORTED, "at_gbt_predict_global_local: n too large");
    DeviceGuard g(global->device);
    hipError_t e = launch_predict(global->desc, feats_global, n, scores, nullptr, false, (hipStream_t)stream);
    if (e == hipSuccess) e = launch_predict(local->desc, feats_local, n, scores, nullptr, true, (hipStream_t)stream);
    return finish_launch(e, "at_gbt_predict_global_local");
}

at_status at_chains_create(at_space_t space, int64_t chain0, int64_t n_chains, int topk, uint64_t seed,
                           at_chains_t* out) {
    if (!out) return fail(AT_E_INVALID, "at_chains_create: out is NULL");
    *out = nullptr;
    if (!space) return fail(AT_E_INVALID, "at_chains_create: NULL space");
    if (chain0 < 0 || n_chains < 0) return fail(AT_E_INVALID, "at_chains_create: negative chain range");
    if (chain0 + n_chains > ((int64_t)1 << 32)) return fail(AT_E_UNSUPPORTED, "at_chains_create: chain ids must fit 32 bits");
    if (topk < 1 || topk > 64) return fail(AT_E_INVALID, "at_chains_create: topk out of [1, 64]");
    if (space->n_spaces > 1 && n_chains != space->chain_offsets.back())
        return fail(AT_E_INVALID, "at_chains_create: n_chains must equal the set's last chain offset");
    at_chains_s* ch = new (std::nothrow) at_chains_s();
    if (!ch) return fail(AT_E_OOM, "at_chains_create: host allocation");
    ch->device = current_device();
    ch->chain0 = chain0;
    ch->n_chains = n_chains;
    ch->topk = topk;
    ch->seed = seed;
    ch->n_spaces = space->n_spaces;
    ch->tmpl = space->api_tmpl;
    at_status st;
    if ((st = alloc_zero(ch->d_knobs, (size_t)n_chains * MAX_KNOBS * 2)) != AT_OK ||
        (st = alloc_zero(ch->d_score, (size_t)n_chains * 4)) != AT_OK ||
        (st = alloc_zero(ch->d_top, (size_t)n_chains * topk * sizeof(at_entry))) != AT_OK ||
        (st = upload(ch->d_descs, space->descs.data(), space->descs.size())) != AT_OK) {
        at_chains_destroy(ch);
        return st;
    }
    if (space->n_spaces > 1) {
        st = upload(ch->d_offsets, space->chain_offsets.data(), space->chain_offsets.size());
    } else {
        const int64_t offs[2] = {0, INT64_MAX};
        st = upload(ch->d_offsets, offs, 2);
    }
    if (st != AT_OK) {
        at_chains_destroy(ch);
        return st;
    }
    *out = ch;
    return AT_OK;
}

void at_chains_destroy(at_chains_t chains) {
    if (!chains) return;
    DeviceGuard g(chains->device);
    release(chains->d_knobs);
    release(chains->d_score);
    release(chains->d_top);
    release(chains->d_descs);
    release(chains->d_offsets);
    release(chains->d_cand);
    release(chains->d_meta);
    release(chains->d_fg);
    release(chains->d_v);
    release(chains->d_tw);
    release(chains->d_fr);
    release(chains->d_vg);
    release(chains->d_twg);
    for (auto& pool : chains->events)
        for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    delete chains;
}

at_status at_sa_set_profiling(at_chains_t chains, int enable) {
    if (!chains) return fail(AT_E_INVALID, "at_sa_set_profiling: NULL chains");
    chains->profiling = enable != 0;
    return AT_OK;
}

at_status at_sa_kernel_times(at_chains_t chains, double* tree_ms, int64_t* tree_launches, double* chain_ms,
                             int64_t* chain_launches) {
    if (!chains) return fail(AT_E_INVALID, "at_sa_kernel_times: NULL chains");
    DeviceGuard g(chains->device);
    double total[2] = {0.0, 0.0};
    for (int kind = 0; kind < 2; ++kind) {
        const std::vector<hipEvent_t>& pool = chains->events[kind];
        for (size_t i = 0; i + 1 < chains->events_used[kind]; i += 2) {
            hipError_t e = hipEventSynchronize(pool[i + 1]);
            if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
            float ms = 0.0f;
            e = hipEventElapsedTime(&ms, pool[i], pool[i + 1]);
            if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
            total[kind] += ms;
        }
    }
    if (tree_ms) *tree_ms = total[0];
    if (tree_launches) *tree_launches = (int64_t)(chains->events_used[0] / 2);
    if (chain_ms) *chain_ms = total[1];
    if (chain_launches) *chain_launches = (int64_t)(chains->events_used[1] / 2);
    return AT_OK;
}

// Argument checks shared by the two selection entry points; AT_OK with
// *nothing set when there is nothing to pick.
static at_status select_args(const char* fn, at_space_t space, const at_entry* cand, int64_t n_cand, int pool,
                             int n_greedy, float alpha, int n_random, at_entry* out, bool* nothing) {
    const std::string f(fn);
    *nothing = false;
    if (!space) return fail(AT_E_INVALID, f + ": NULL space");
    if (space->n_spaces != 1) return fail(AT_E_INVALID, f + ": takes a single space, not a set");
    if (n_cand < 0 || pool < 0 || n_greedy < 0 || n_random < 0) return fail(AT_E_INVALID, f + ": negative size");
    if (n_cand > 0 && !cand) return fail(AT_E_INVALID, f + ": NULL candidates");
    if (pool > select_pool_max()) return fail(AT_E_UNSUPPORTED, f + ": pool above 1024");
    if ((int64_t)n_greedy + n_random > select_pick_max()) return fail(AT_E_UNSUPPORTED, f + ": more than 2048 picks");
    if (!std::isfinite(alpha)) return fail(AT_E_INVALID, f + ": alpha must be finite");
    const SpaceDesc& d = space->descs[0];
    for (int j = 0; j < d.n_knobs; ++j)
        if (d.knob_size[j] > 65536u) return fail(AT_E_UNSUPPORTED, f + ": a knob has more than 65536 values");
    if (n_greedy + n_random == 0) {
        *nothing = true;
        return AT_OK;
    }
    if (!out) return fail(AT_E_INVALID, f + ": NULL output");
    if (n_cand > ((int64_t)1 << 40)) return fail(AT_E_UNSUPPORTED, f + ": too many candidates");
    return AT_OK;
}

at_status at_select_batch(at_space_t space, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                          float alpha, int n_random, uint64_t seed, at_entry* out, at_stream_t stream) {
    bool nothing = false;
    const at_status st = select_args("at_select_batch", space, cand, n_cand, pool, n_greedy, alpha, n_random, out,
                                     &nothing);
    if (st != AT_OK || nothing) return st;
    DeviceGuard g(space->device);
    return finish_launch(launch_select(*space, cand, n_cand, pool, n_greedy, alpha, n_random, seed, out,
                                       (hipStream_t)stream, nullptr),
                         "at_select_batch");
}

at_status at_select_batch_noalloc(at_space_t space, const at_entry* cand, int64_t n_cand, int pool, int n_greedy,
                                  float alpha, int n_random, uint64_t seed, at_entry* out, at_stream_t stream) {
    bool nothing = false;
    const at_status st = select_args("at_select_batch_noalloc", space, cand, n_cand, pool, n_greedy, alpha,
                                     n_random, out, &nothing);
    if (st != AT_OK || nothing) return st;
    if (select_scratch_entries(n_cand, pool) > select_scratch_max_entries())
        return fail(AT_E_UNSUPPORTED, "at_select_batch_noalloc: ceil(n_cand / 2048) * max(pool, 1) rounded up to "
                                      "a power of two exceeds the scratch limit of " +
                                      std::to_string(select_scratch_max_entries()) + " entries");
    DeviceGuard g(space->device);
    at_entry* scratch = nullptr;
    const hipError_t e = select_scratch_ptr(space->device, &scratch);
    if (e != hipSuccess) return hip_fail(e, "at_select_batch_noalloc: hipGetSymbolAddress");
    return finish_launch(launch_select(*space, cand, n_cand, pool, n_greedy, alpha, n_random, seed, out,
                                       (hipStream_t)stream, scratch),
                         "at_select_batch_noalloc");
}

at_status at_chains_set_path(at_chains_t chains, int path) {
    if (!chains) return fail(AT_E_INVALID, "at_chains_set_path: NULL chains");
    if (path != AT_SA_PATH_AUTO && path != AT_SA_PATH_TREES && path != AT_SA_PATH_LOCAL)
        return fail(AT_E_INVALID, "at_chains_set_path: unknown path");
    chains->path = path;
    return AT_OK;
}

at_status at_chains_last_path(at_chains_t chains, int* path) {
    if (!chains || !path) return fail(AT_E_INVALID, "at_chains_last_path: NULL argument");
    *path = chains->last_path;
    return AT_OK;
}

at_status at_chains_last_plan(at_chains_t chains, int64_t info[8]) {
    if (!chains || !info) return fail(AT_E_INVALID, "at_chains_last_plan: NULL argument");
    for (int i = 0; i < 8; ++i) info[i] = chains->last_plan[i];
    return AT_OK;
}

at_status at_chains_step(at_chains_t chains, uint64_t* step_abs) {
    if (!chains || !step_abs) return fail(AT_E_INVALID, "at_chains_step: NULL argument");
    *step_abs = chains->step_abs;
    return AT_OK;
}

at_status at_sa_thresholds(uint64_t seed, int64_t chain0, int64_t n_chains, uint64_t step_base, int steps,
                           float* thr) {
    if (steps < 1 || n_chains < 0 || chain0 < 0) return fail(AT_E_INVALID, "at_sa_thresholds: bad sizes");
    if (n_chains > 0 && !thr) return fail(AT_E_INVALID, "at_sa_thresholds: NULL output");
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int64_t c = 0; c < n_chains; ++c) {
        const uint32_t chain = (uint32_t)(chain0 + c);
        for (int s = 0; s < steps; ++s) {
            const U4 r = philox(k0, k1, U4{chain, (uint32_t)(step_base + (uint64_t)s), 0u, 0u});
            const double T = steps == 1 ? 0.0 : 1.0 - (double)s / (double)(steps - 1);
            const double u = ((double)r.z + 0.5) / 4294967296.0;
            thr[c * steps + s] = (float)(T * std::log(u));
        }
    }
    return AT_OK;
}

static at_status sa_run_impl(at_space_t space, at_ensemble_t ens, at_ensemble_t global, at_chains_t chains,
                             int steps, const float* thr, at_entry* best, at_entry* trace, at_stream_t stream,
                             const char* fn) {
    const std::string f(fn);
    if (!space || !ens || !chains) return fail(AT_E_INVALID, f + ": NULL handle");
    if (steps < 0) return fail(AT_E_INVALID, f + ": steps < 0");
    if (space->n_spaces != chains->n_spaces || space->api_tmpl != chains->tmpl)
        return fail(AT_E_INVALID, f + ": chains were created for another space");
    if (space->n_spaces > 1 && chains->n_chains != space->chain_offsets.back())
        return fail(AT_E_INVALID, f + ": chain count does not match the space set");
    if (ens->desc.n_features != space->descs[0].n_features)
        return fail(AT_E_MISMATCH, f + ": ensemble and space feature counts differ");
    if (global && global->desc.n_features != RELATION_FEATURES)
        return fail(AT_E_MISMATCH, f + ": the global model must read the 192 context relation features");
    if (chains->n_chains > 0 && !best) return fail(AT_E_INVALID, f + ": NULL best");
    if (steps > 0 && chains->n_chains > 0 && !thr) return fail(AT_E_INVALID, f + ": NULL thr");
    if (chains->step_abs + (uint64_t)steps > ((uint64_t)1 << 32))
        return fail(AT_E_UNSUPPORTED, f + ": step counter must fit 32 bits");
    DeviceGuard g(chains->device);
    const bool init = !chains->initialised;
    // path: chain-local when its plan fits and one workgroup streams at most
    // LOCAL_AUTO_BYTES per step, else tree-partitioned; Eq. 4 runs take the
    // tree-partitioned path
    LocalPlan pl;
    const bool local_fits = !global && chains->n_chains > 0 && plan_local(*space, ens->desc, *chains, pl);
    int path = chains->path;
    if (path == AT_SA_PATH_AUTO)
        path = (local_fits && pl.round_bytes <= LOCAL_AUTO_BYTES) ? AT_SA_PATH_LOCAL : AT_SA_PATH_TREES;
    if (path == AT_SA_PATH_LOCAL && global)
        return fail(AT_E_UNSUPPORTED, f + ": two-model (Eq. 4) runs take the tree-partitioned path");
    if (path == AT_SA_PATH_LOCAL && chains->n_chains > 0 && !local_fits)
        return fail(AT_E_UNSUPPORTED, f + ": the chain-local plan does not fit one workgroup's LDS");
    hipError_t e = path == AT_SA_PATH_LOCAL
                       ? launch_sa_local(*space, ens->desc, *chains, pl, steps, init, thr, best, trace,
                                         (hipStream_t)stream)
                       : launch_sa_tp(*space, ens->desc, global ? &global->desc : nullptr, *chains, steps, init, thr,
                                      best, trace, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, fn);
    chains->last_path = path;
    const int64_t plan[8] = {pl.cpb, pl.threads, pl.grid, pl.ct, (pl.resident || pl.tail) ? 0 : pl.n_chunks,
                             pl.tail ? 2 : pl.gather, (int64_t)pl.lds_bytes, (int64_t)pl.round_bytes};
    // the tree-partitioned launcher records its own plan
    if (path == AT_SA_PATH_LOCAL)
        for (int i = 0; i < 8; ++i) chains->last_plan[i] = plan[i];
    else if (chains->n_chains == 0)
        for (int i = 0; i < 8; ++i) chains->last_plan[i] = 0;
    chains->initialised = true;
    chains->step_abs += (uint64_t)steps;
    return AT_OK;
}

at_status at_sa_run(at_space_t space, at_ensemble_t ens, at_chains_t chains, int steps, const float* thr,
                    at_entry* best, at_stream_t stream) {
    return sa_run_impl(space, ens, nullptr, chains, steps, thr, best, nullptr, stream, "at_sa_run");
}

at_status at_sa_run_traced(at_space_t space, at_ensemble_t ens, at_chains_t chains, int steps, const float* thr,
                           at_entry* best, at_entry* trace, at_stream_t stream) {
    if (steps > 0 && chains && chains->n_chains > 0 && !trace) return fail(AT_E_INVALID, "at_sa_run_traced: NULL trace");
    return sa_run_impl(space, ens, nullptr, chains, steps, thr, best, trace, stream, "at_sa_run_traced");
}

at_status at_sa_run_global_local(at_space_t space, at_ensemble_t global, at_ensemble_t local, at_chains_t chains,
                                 int steps, const float* thr, at_entry* best, at_entry* trace, at_stream_t stream) {
    if (!global) return fail(AT_E_INVALID, "at_sa_run_global_local: NULL global model");
    return sa_run_impl(space, local, global, chains, steps, thr, best, trace, stream, "at_sa_run_global_local");
}

at_status at_chains_export(at_chains_t chains, uint64_t* cur_cfg, float* cur_score, at_stream_t stream) {
    if (!chains) return fail(AT_E_INVALID, "at_chains_export: NULL chains");
    if (!chains->initialised) return fail(AT_E_INVALID, "at_chains_export: chains not initialised (run at_sa_run first)");
    DeviceGuard g(chains->device);
    return finish_launch(launch_export(*chains, cur_cfg, cur_score, (hipStream_t)stream), "at_chains_export");
}

}  // extern "C"
