// Device helpers shared by the kernels: wavefront-aggregated list appends and
// the structural change-list propagation rule.
#pragma once

#include "sscater_internal.h"

namespace ssc {

typedef float f4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63u); }

// Structural propagation of changed cells to the next layer's list, in two
// phases for latency hiding.  Cell (i, j) of the grid (t.Hin x t.Win) feeds
// output ((i - m + 1)/s, (j - n + 1)/s) through tap (m, n) when both quotients
// are integral and inside (t.Hout x t.Wout): the scatter target of Eq. 2
// generalised to stride s, and the downsampling rule of Alg. 1 for s = 2.
// Each cell is handled by G lanes that share its 9 tap slots (slot = sub +
// it*G).  prop_issue stamps every target with `epoch` (atomicMax: the lane
// that moves a stamp owns the target); prop_finish (later, after unrelated
// work) counts the pairs and appends the owned targets of the wavefront to
// list segment `shard` with a single atomic.
// Both must be reached by every lane of the wavefront.
template <int G>
struct PropBatch {
    static constexpr int ITERS = (9 + G - 1) / G;
    int q[ITERS];
    uint32_t old[ITERS];   // stamp before this lane's atomic (owner iff < epoch)
};

// cell: a valid cell of the source grid (used for addressing even when
// inactive); active: whether the cell really changed.
// UNCOND = true: every lane issues its atomic unconditionally so that no
// branch joins on the returned value (a join would make the compiler wait for
// it right there).  A slot without a target stamps a clamped cell next to
// `cell` with 0, which never changes a stamp (stamps only grow and epochs
// start at 1); the addresses stay spread over the grid.  Use it where most
// lanes are active.  UNCOND = false: inactive lanes issue nothing.
template <int G, bool UNCOND>
__device__ __forceinline__ void prop_issue(const PropTarget& t, int cell, bool active, int sub, uint32_t epoch,
                                           PropBatch<G>& pb) {
    const int img = cell / (t.Hin * t.Win), loc = cell - img * (t.Hin * t.Win);
    const int i = loc / t.Win, j = loc - (loc / t.Win) * t.Win;
    const int obase = img * (t.Hout * t.Wout);
#pragma unroll
    for (int it = 0; it < PropBatch<G>::ITERS; ++it) {
        const int k = sub + it * G;
        const int m = k / 3, n = k - 3 * (k / 3);
        int rn = i - m + 1, cn = j - n + 1;
        bool ok = active && k < 9;
        if (t.stride == 2) {
            ok = ok && ((rn | cn) & 1) == 0;
            rn >>= 1;
            cn >>= 1;
        }
        ok = ok && rn >= 0 && rn < t.Hout && cn >= 0 && cn < t.Wout;
        const int q = obase + min(max(rn, 0), t.Hout - 1) * t.Wout + min(max(cn, 0), t.Wout - 1);
        pb.q[it] = ok ? q : -1;
        if (UNCOND) {
            pb.old[it] = atomicMax(&t.stamp[q], ok ? epoch : 0u);
        } else if (ok) {
            // pb.old is read only where q >= 0; leaving it unset on the other
            // path avoids a register copy that would wait for the atomic
            pb.old[it] = atomicMax(&t.stamp[q], epoch);
        }
    }
}

template <int G>
__device__ __forceinline__ void prop_finish(const PropTarget& t, uint32_t epoch, int shard, PropBatch<G>& pb) {
    constexpr int IT = PropBatch<G>::ITERS;
    const int lane = lane_id();
    const unsigned long long lt = (1ull << lane) - 1ull;
    unsigned long long ob[IT];
    bool own[IT];
    int pairs = 0, tot = 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        own[it] = pb.q[it] >= 0 && pb.old[it] < epoch;
        pairs += (int)__popcll(__ballot(pb.q[it] >= 0));
        ob[it] = __ballot(own[it]);
        tot += (int)__popcll(ob[it]);
    }
    int base = 0;
    if (lane == 0) {
        if (tot) base = atomicAdd(t.count + shard * CSTRIDE, tot);
        if (pairs) atomicAdd(t.pairs + (shard * PSPREAD + (int)(blockIdx.x & (PSPREAD - 1))) * CSTRIDE, pairs);
    }
    if (tot == 0) return;
    base = __shfl(base, 0);
    int32_t* seg = t.list + (size_t)shard * t.seg;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        if (own[it]) seg[base + (int)__popcll(ob[it] & lt)] = pb.q[it];
        base += (int)__popcll(ob[it]);
    }
}

// Active-set words (sparse backbones): see MembTarget.
__device__ __forceinline__ bool memb_now(uint64_t w) { return (uint32_t)w != 0u; }

__device__ __forceinline__ bool memb_prev(uint64_t w, uint32_t epoch) {
    return (uint32_t)(w >> 33) == (epoch & 0x7FFFFFFFu) ? ((w >> 32) & 1ull) != 0ull : memb_now(w);
}

// Counts of the next regular layer: +-1 at every output site whose receptive
// field holds `cell` (the same stride rule as the change lists), in two
// halves like the propagation: memb_issue computes the targets and loads
// their words (from clamped, always valid addresses, also where `on` is
// false, so that no branch joins on the loads), memb_finish compare-and-swaps
// them.  A swap that lost to another lane or workgroup goes round again; all
// of a lane's pending targets go round together, so a round costs one round
// trip however many of them collided.
struct MembBatch {
    unsigned long long old[9];   // the targets' words as loaded
    uint32_t todo;               // bit k: target k exists and is to be updated
};

// Target k of `cell` (clamped to the grid) and whether it exists.
__device__ __forceinline__ unsigned long long* memb_target(const MembTarget& t, int cell, int hin, int win, int k,
                                                            bool& ok) {
    const int img = cell / (hin * win), loc = cell - img * (hin * win);
    const int i = loc / win, j = loc - (loc / win) * win;
    int rn = i - k / 3 + 1, cn = j - k % 3 + 1;
    ok = true;
    if (t.stride == 2) {
        ok = ((rn | cn) & 1) == 0;
        rn >>= 1;
        cn >>= 1;
    }
    ok = ok && rn >= 0 && rn < t.Hout && cn >= 0 && cn < t.Wout;
    return reinterpret_cast<unsigned long long*>(t.memb) + (size_t)img * t.Hout * t.Wout +
           (size_t)min(max(rn, 0), t.Hout - 1) * t.Wout + min(max(cn, 0), t.Wout - 1);
}

__device__ __forceinline__ void memb_issue(const MembTarget& t, int cell, int hin, int win, bool on, MembBatch& mb) {
    mb.todo = 0u;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        bool ok;
        unsigned long long* p = memb_target(t, cell, hin, win, k, ok);
        if (on && ok) mb.todo |= 1u << k;
        mb.old[k] = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The word after adding `delta` to the count; the first change of a stride
// (epoch ep) records whether the site was active before it.
__device__ __forceinline__ unsigned long long memb_next(unsigned long long w, int delta, unsigned long long ep) {
    const uint32_t cnt = (uint32_t)w;
    const unsigned long long was = ((w >> 33) == ep) ? ((w >> 32) & 1ull) : (cnt != 0u ? 1ull : 0ull);
    return (ep << 33) | (was << 32) | (unsigned long long)(uint32_t)(cnt + (uint32_t)delta);
}

// memb_finish in two halves, so that the first swaps' round trip can overlap
// another (memb_swap issues them, memb_settle retries the lost ones); cell,
// hin, win: as given to memb_issue.
__device__ __forceinline__ void memb_swap(const MembTarget& t, int cell, int hin, int win, const MembBatch& mb,
                                          int delta, uint32_t epoch, unsigned long long (&got)[9]) {
    const unsigned long long ep = epoch & 0x7FFFFFFFu;
#pragma unroll
    for (int k = 0; k < 9; ++k) got[k] = mb.old[k];
    if (mb.todo == 0u) return;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        bool ok;
        unsigned long long* p = memb_target(t, cell, hin, win, k, ok);
        if ((mb.todo >> k) & 1u) got[k] = atomicCAS(p, mb.old[k], memb_next(mb.old[k], delta, ep));
    }
}

__device__ __forceinline__ void memb_settle(const MembTarget& t, int cell, int hin, int win, MembBatch& mb, int delta,
                                            uint32_t epoch, const unsigned long long (&got0)[9]) {
    const unsigned long long ep = epoch & 0x7FFFFFFFu;
    uint32_t todo = 0u;
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        if (((mb.todo >> k) & 1u) && got0[k] != mb.old[k]) todo |= 1u << k;   // lost: retry from the word it found
        mb.old[k] = got0[k];
    }
    if (todo == 0u) return;
    unsigned long long* ptr[9];
#pragma unroll
    for (int k = 0; k < 9; ++k) {
        bool ok;
        ptr[k] = memb_target(t, cell, hin, win, k, ok);
    }
    while (todo) {
        unsigned long long got[9];
#pragma unroll
        for (int k = 0; k < 9; ++k)
            got[k] = (todo >> k) & 1u ? atomicCAS(ptr[k], mb.old[k], memb_next(mb.old[k], delta, ep)) : 0ull;
        uint32_t lost = 0u;
#pragma unroll
        for (int k = 0; k < 9; ++k) {
            if (((todo >> k) & 1u) && got[k] != mb.old[k]) lost |= 1u << k;
            mb.old[k] = got[k];
        }
        todo = lost;
    }
}

// cell, hin, win: as given to memb_issue.
__device__ __forceinline__ void memb_finish(const MembTarget& t, int cell, int hin, int win, MembBatch& mb, int delta,
                                            uint32_t epoch) {
    unsigned long long got[9];
    memb_swap(t, cell, hin, win, mb, delta, epoch, got);
    memb_settle(t, cell, hin, win, mb, delta, epoch, got);
}

__device__ __forceinline__ void memb_spread(const MembTarget& t, int cell, int hin, int win, int delta,
                                            uint32_t epoch) {
    MembBatch mb;
    memb_issue(t, cell, hin, win, true, mb);
    memb_finish(t, cell, hin, win, mb, delta, epoch);
}

// prop_finish in two halves, so that the counter's round trip overlaps other
// work: prop_reserve counts the owned targets and takes their list positions
// (the atomic's result is not waited for), prop_write stores the entries.
template <int G>
struct PropSlots {
    static constexpr int IT = PropBatch<G>::ITERS;
    unsigned long long ob[IT];
    bool own[IT];
    int base, tot;
};

template <int G>
__device__ __forceinline__ void prop_reserve(const PropTarget& t, uint32_t epoch, int shard, const PropBatch<G>& pb,
                                             PropSlots<G>& ps) {
    constexpr int IT = PropBatch<G>::ITERS;
    int pairs = 0;
    ps.tot = 0;
    ps.base = 0;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        ps.own[it] = pb.q[it] >= 0 && pb.old[it] < epoch;
        pairs += (int)__popcll(__ballot(pb.q[it] >= 0));
        ps.ob[it] = __ballot(ps.own[it]);
        ps.tot += (int)__popcll(ps.ob[it]);
    }
    if (lane_id() == 0) {
        if (ps.tot) ps.base = atomicAdd(t.count + shard * CSTRIDE, ps.tot);
        if (pairs) atomicAdd(t.pairs + (shard * PSPREAD + (int)(blockIdx.x & (PSPREAD - 1))) * CSTRIDE, pairs);
    }
}

template <int G>
__device__ __forceinline__ void prop_write(const PropTarget& t, int shard, const PropBatch<G>& pb, PropSlots<G>& ps) {
    constexpr int IT = PropBatch<G>::ITERS;
    if (ps.tot == 0) return;
    const unsigned long long lt = (1ull << lane_id()) - 1ull;
    int base = __shfl(ps.base, 0);
    int32_t* seg = t.list + (size_t)shard * t.seg;
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        if (ps.own[it]) seg[base + (int)__popcll(ps.ob[it] & lt)] = pb.q[it];
        base += (int)__popcll(ps.ob[it]);
    }
}

// fp32 -> bf16 bits, round to nearest even (finite values).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// Z update and next-layer delta row of one lane: output cell q, output
// channels co0 .. co0+3 (fp32 Z_new = Z_old + D; delta phi(Z_new) -
// phi(Z_old), or the bf16 pair [bf16(phi(Z_new)) | bf16(phi(Z_old))]).
// Sparse backbones: now / prev say whether the site is active in this and
// in the previous stride; an inactive site's output is zero.
template <int COUT, bool BF16>
__device__ __forceinline__ void epilogue4(const LayerArgs& a, int q, int co0, const f4v o, const f4v d,
                                          bool now = true, bool prev = true) {
    f4v zn;
    zn.x = o.x + d.x;
    zn.y = o.y + d.y;
    zn.z = o.z + d.z;
    zn.w = o.w + d.w;
    *reinterpret_cast<f4v*>(a.Z + (size_t)q * COUT + co0) = zn;
    if (!a.delta_out) return;
    f4v yo = o, yn = zn;
    if (a.relu) {
        yo.x = fmaxf(yo.x, 0.f); yo.y = fmaxf(yo.y, 0.f); yo.z = fmaxf(yo.z, 0.f); yo.w = fmaxf(yo.w, 0.f);
        yn.x = fmaxf(yn.x, 0.f); yn.y = fmaxf(yn.y, 0.f); yn.z = fmaxf(yn.z, 0.f); yn.w = fmaxf(yn.w, 0.f);
    }
    if (!prev) yo = f4v{0.f, 0.f, 0.f, 0.f};
    if (!now) yn = f4v{0.f, 0.f, 0.f, 0.f};
    char* drow = static_cast<char*>(a.delta_out) + (size_t)q * (4 * COUT);
    if constexpr (BF16) {
        uint2 pn, po;
        pn.x = f32_to_bf16_bits(yn.x) | (f32_to_bf16_bits(yn.y) << 16);
        pn.y = f32_to_bf16_bits(yn.z) | (f32_to_bf16_bits(yn.w) << 16);
        po.x = f32_to_bf16_bits(yo.x) | (f32_to_bf16_bits(yo.y) << 16);
        po.y = f32_to_bf16_bits(yo.z) | (f32_to_bf16_bits(yo.w) << 16);
        *reinterpret_cast<uint2*>(drow + co0 * 2) = pn;
        *reinterpret_cast<uint2*>(drow + COUT * 2 + co0 * 2) = po;
    } else {
        f4v dy;
        dy.x = yn.x - yo.x;
        dy.y = yn.y - yo.y;
        dy.z = yn.z - yo.z;
        dy.w = yn.w - yo.w;
        *reinterpret_cast<f4v*>(drow + co0 * 4) = dy;
    }
}

// ---- rings of LDS stages filled by asynchronous global->LDS copies ----

// s_waitcnt with only the vector-memory count limited to n.
template <int n>
__device__ __forceinline__ void wait_vm() {
    static_assert(n >= 0 && n < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14));
}

// Workgroup barrier without a memory fence.  __syncthreads() also drains
// every outstanding global access and LDS copy (vmcnt(0)), which would wait
// for the copies of the later chunks too.  Here each thread first waits for
// its own copies of the chunk it needs (wait_vm), and its LDS reads of the
// previous chunk have completed before their matrix instructions ran, so the
// hardware barrier makes the stage safe once this wavefront's own LDS reads
// have completed; the empty asm statements keep the compiler from moving
// memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("" ::: "memory");
    // this wavefront's LDS reads are complete (lgkmcnt(0), no vmcnt limit)
    __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// wait_vm for a count known once the chunk loop is unrolled
__device__ __forceinline__ void wait_vm_n(int n) {
    switch (n) {
        case 0: wait_vm<0>(); break;
        case 4: wait_vm<4>(); break;
        case 6: wait_vm<6>(); break;
        case 8: wait_vm<8>(); break;
        case 12: wait_vm<12>(); break;
        case 16: wait_vm<16>(); break;
        case 18: wait_vm<18>(); break;
        case 24: wait_vm<24>(); break;
        case 32: wait_vm<32>(); break;
        default: wait_vm<0>(); break;
    }
}

__device__ __forceinline__ void copy16(const void* src, void* lds) {
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}

__device__ __forceinline__ void flag_error(int32_t* err, int bit) {
    *(volatile int32_t*)err = bit;
}

}  // namespace ssc
