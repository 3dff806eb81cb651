// Chain bookkeeping shared by the annealing kernels: knob vectors packed as
// u16, the space of a chain in a space set, and insertion into a chain's
// best list (Section 3.3: every scored candidate is offered; entries are
// ordered by score descending, then configuration index ascending, with
// distinct indices).
#pragma once

#include "at_device.h"

namespace at {
namespace dev {

// Workgroup barrier that orders LDS accesses only: each wave's own LDS
// operations complete before it arrives; global loads stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ __forceinline__ int space_of(const int64_t* offsets, int n_spaces, int64_t c) {
    int w = 0;
    while (w + 1 < n_spaces && offsets[w + 1] <= c) ++w;
    return w;
}

// A chain's knob vector: MAX_KNOBS u16 (24 bytes, three 8-byte words).
static_assert(MAX_KNOBS == 12, "knob vectors move as three 8-byte words");
__device__ __forceinline__ void load_knob_words(const uint16_t* p, int64_t c, uint2 (&w)[3]) {
    const uint2* q = reinterpret_cast<const uint2*>(p) + 3 * c;
    w[0] = q[0];
    w[1] = q[1];
    w[2] = q[2];
}

__device__ __forceinline__ void unpack_knobs(const uint2 (&w)[3], uint32_t (&kv)[MAX_KNOBS]) {
    const uint32_t pw[6] = {w[0].x, w[0].y, w[1].x, w[1].y, w[2].x, w[2].y};
#pragma unroll
    for (int j = 0; j < MAX_KNOBS; ++j) kv[j] = (pw[j >> 1] >> (16 * (j & 1))) & 0xffffu;
}

__device__ __forceinline__ void load_knobs(const uint16_t* p, int64_t c, uint32_t (&kv)[MAX_KNOBS]) {
    uint2 w[3];
    load_knob_words(p, c, w);
    unpack_knobs(w, kv);
}

__device__ __forceinline__ void store_knobs(uint16_t* p, int64_t c, const uint32_t (&kv)[MAX_KNOBS]) {
    uint2* w = reinterpret_cast<uint2*>(p) + 3 * c;
    w[0] = make_uint2(kv[0] | (kv[1] << 16), kv[2] | (kv[3] << 16));
    w[1] = make_uint2(kv[4] | (kv[5] << 16), kv[6] | (kv[7] << 16));
    w[2] = make_uint2(kv[8] | (kv[9] << 16), kv[10] | (kv[11] << 16));
}

__device__ __forceinline__ bool precedes(float sa, uint64_t ca, float sb, uint64_t cb) {
    return sa > sb || (sa == sb && ca < cb);
}

// Per-chain record shared between the chain's owner lane and its group of
// 16 lanes through LDS.
struct ChainRec {
    uint64_t cfg;
    float score;
    uint32_t count;
    float kth_score;
    uint32_t qual;
    uint64_t kth_cfg;
    uint32_t nx[MAX_KNOBS / 2];   // proposed knob values, packed in pairs
    // chain-local path, ahead of time: the next candidate if this one is
    // rejected (nx holds the one if it is accepted), and which of the two
    // feature rows the next round uses (0: accepted, 1: rejected)
    uint32_t nxb[MAX_KNOBS / 2];
    uint32_t sel;
    uint64_t cfga, cfgb;          // configuration indices of nx and nxb
    float thr;                    // the next round's Metropolis threshold
    // drawn moves by step parity (knob, value, knob weight) and the scored
    // candidates waiting for their offer, by round parity
    int32_t mvj[2];
    uint32_t mvv[2];
    uint64_t mvr[2];
    uint64_t pcfg[2];
    float pscore[2];
    // chain-local fast rounds, by round parity: the round's two candidates
    // (outcome 0 after an accept, 1 after a reject; knobs packed in pairs,
    // index), the outcome that holds the round's candidate, and the current
    // configuration the round starts from
    uint32_t snx[2][2][MAX_KNOBS / 2];
    uint64_t scfg[2][2];
    uint32_t ssel[2];
    uint32_t curk[2][MAX_KNOBS / 2];
    uint64_t curcfg[2];
};

// Offers (cfg, sc) to the best list of one chain held in LDS, with the 16
// lanes r = 0..15 of its group (entries are ordered by score descending then
// index ascending, distinct indices, at most k <= 64).  Lane r looks after
// entries r, r+16, r+32, r+48.  A wave ballot gives whether the index is
// already listed and how many entries precede the new one (its position);
// the entries from that position on then move down by one.  All lanes of
// the wave must call this (the ballots are wave-wide); gm selects the
// group's 16 bits of a ballot mask and `active` the lanes of a group whose
// chain offers.
// Rec: any record with cfg, score, count, kth_score and kth_cfg.
// gout / gmeta (optional): the chain's list and ChainMeta in global memory;
// every entry the offer changes and the list's new count and k-th entry are
// also written there by the lane that makes them.
template <class Rec>
__device__ __forceinline__ void group_offer(at_entry* list, Rec& rec, int k, int r, uint64_t gm, bool active,
                                            at_entry* gout = nullptr, ChainMeta* gmeta = nullptr) {
    const uint64_t cfg = rec.cfg;
    const float sc = rec.score;
    const int count = active ? (int)rec.count : 0;
    at_entry old[4], prev[4];
    bool dup = false;
    uint32_t pre = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = r + 16 * u;
        if (active && i < count) {
            old[u] = list[i];
            dup |= old[u].cfg == cfg;
            pre |= precedes(old[u].score, old[u].cfg, sc, cfg) ? (1u << u) : 0u;
        }
        if (active && i > 0 && i <= count && i < k) prev[u] = list[i - 1];
    }
    const bool any_dup = (__ballot(dup) & gm) != 0;
    int pos = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) pos += __popcll(__ballot((pre >> u) & 1u) & gm);
    if (!active || any_dup) return;
    // new list: entries before pos stay, the new entry goes to pos, later
    // entries move down one place, the last one drops out when the list is full
    const int n_new = count < k ? count + 1 : k;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int i = r + 16 * u;
        if (i >= pos && i < n_new) {
            at_entry e;
            if (i == pos) {
                e.cfg = cfg;
                e.score = sc;
                e.flag = 1u;
            } else {
                e = prev[u];
            }
            list[i] = e;
            if (gout) gout[i] = e;
            if (i == n_new - 1) {
                rec.count = (uint32_t)n_new;
                rec.kth_score = e.score;
                rec.kth_cfg = e.cfg;
                if (gmeta) {
                    ChainMeta m;
                    m.count = (uint32_t)n_new;
                    m.kth_score = e.score;
                    m.kth_cfg = e.cfg;
                    *gmeta = m;
                }
            }
        }
    }
}

// One level of four trees: for each tree, right = (node & 0xff) <= x4, node
// becomes the right or left half of its children pair pr, p becomes 2p +
// right (the comparison's carry), then the next feature address
// (node & mask) | fb and pair address nb + 4p.  The compiler does not form
// the carry and the half-word select from plain code.  A VALU write of VCC
// is read two or more instructions later (gfx950 wait states): the first
// compare is followed by s_nop 1, the others by the previous tree's address
// instructions.
// Operands: 0-3 node, 4-7 p, 8-11 feature address, 12-15 pair address,
// 16-19 x4, 20-23 pr, 24 mask, 25 fb, 26-29 nb.
#define AT_WALK4_ASM                                                                                       \
    "v_cmp_le_u32_sdwa vcc, %0, %16 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "s_nop 1\n\t"                                                                                          \
    "v_cndmask_b32_sdwa %0, %20, %20, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t" \
    "v_addc_co_u32 %4, vcc, %4, %4, vcc\n\t"                                                               \
    "v_cmp_le_u32_sdwa vcc, %1, %17 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %8, %0, %24, %25\n\t"                                                                    \
    "v_lshl_add_u32 %12, %4, 2, %26\n\t"                                                                   \
    "v_cndmask_b32_sdwa %1, %21, %21, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t" \
    "v_addc_co_u32 %5, vcc, %5, %5, vcc\n\t"                                                               \
    "v_cmp_le_u32_sdwa vcc, %2, %18 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %9, %1, %24, %25\n\t"                                                                    \
    "v_lshl_add_u32 %13, %5, 2, %27\n\t"                                                                   \
    "v_cndmask_b32_sdwa %2, %22, %22, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t" \
    "v_addc_co_u32 %6, vcc, %6, %6, vcc\n\t"                                                               \
    "v_cmp_le_u32_sdwa vcc, %3, %19 src0_sel:BYTE_0 src1_sel:DWORD\n\t"                                    \
    "v_and_or_b32 %10, %2, %24, %25\n\t"                                                                   \
    "v_lshl_add_u32 %14, %6, 2, %28\n\t"                                                                   \
    "v_cndmask_b32_sdwa %3, %23, %23, vcc dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_1\n\t" \
    "v_addc_co_u32 %7, vcc, %7, %7, vcc\n\t"                                                               \
    "v_and_or_b32 %11, %3, %24, %25\n\t"                                                                   \
    "v_lshl_add_u32 %15, %7, 2, %29"

}  // namespace dev
}  // namespace at
