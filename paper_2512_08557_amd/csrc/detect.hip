// Changed-cell detector on the input canvas: marks the input change set A_0
// (stamps), writes the input deltas at their cells, updates the canvas and
// propagates A_0 to the first layer's change list.
//
// A cell is changed when its stored feature vector differs bit for bit from
// the canvas (a pillar whose points changed: Sec. III-B and Alg. 1, PFN part).
// Two passes per stride:
//   present  : every pillar of the new list is compared with the canvas and
//              writes its cell's presence word (epoch, row) with a plain store;
//   vanished : every cell of the previous list that is absent from the new
//              list is compared with zero (its pillar disappeared); the same
//              pass checks that every pillar of the new list owns its cell's
//              presence word (two pillars on one cell are an input fault).
// The second pass needs the presence words of the whole first pass, so it is
// a separate launch; for a list sorted by cell, detect_sorted_kernel does both
// in one launch (each workgroup merges its stretch of the two lists).
// Sparse backbones (SPARSE): the pillar set is itself an input, so a pillar
// that appeared or vanished is changed whatever its values, and it moves the
// first layer's active-set counts (memb_spread).
//
// Layout: G = row_bytes / 16 lanes share one feature row, each lane moving 16
// bytes, so a 64-channel fp32 row (256 B) is one fully coalesced 16-lane
// access.  Delta rows (4*C0 bytes at the cell's position): fp32 new - old, or
// for bf16 the pair [new | old] that the layer kernels contract exactly (no
// delta rounding).
#include "device_common.h"

#include <algorithm>

namespace ssc {

// The end of one pass over G-lane rows, shared by every mode: the lanes of a
// row (sub = the lane's piece of it) hold the cell p (pc: p, or 0 when the
// row is inactive) and the 16-byte pieces nv (new) and ov (old) of its
// features; tog: a sparse pillar that appeared or vanished.  A changed row
// writes its delta, the new canvas row and its stamp, and the cell goes to
// the first layer's list.
template <int ROWB, bool BF16, bool SPARSE>
__device__ __forceinline__ void emit_rows(const DetectArgs& a, int p, int pc, bool act, bool tog, uint4 nv, uint4 ov,
                                          int shard, bool vanish) {
    constexpr int G = ROWB / 16;
    constexpr int DROWB = BF16 ? 2 * ROWB : ROWB;   // delta row bytes
    const int lane = lane_id();
    const int sub = lane % G;
    const int gbase = lane - sub;
    const bool d = act && (tog || nv.x != ov.x || nv.y != ov.y || nv.z != ov.z || nv.w != ov.w);
    const unsigned long long bal = __ballot(d);
    const unsigned long long gm = (G == 64 ? ~0ull : ((1ull << G) - 1ull)) << gbase;
    const bool gd = (bal & gm) != 0ull;
    // stamp the first layer's footprint while the rows are written
    PropBatch<G> pb;
    prop_issue<G, false>(a.next, pc, gd, sub, a.epoch, pb);
    if (gd) {
        char* xrow = static_cast<char*>(a.X) + (size_t)pc * ROWB + sub * 16;
        char* drow = static_cast<char*>(a.delta0) + (size_t)p * DROWB;
        if (BF16) {
            *reinterpret_cast<uint4*>(drow + sub * 16) = nv;
            *reinterpret_cast<uint4*>(drow + ROWB + sub * 16) = ov;
        } else {
            f4v dn;
            dn.x = __uint_as_float(nv.x) - __uint_as_float(ov.x);
            dn.y = __uint_as_float(nv.y) - __uint_as_float(ov.y);
            dn.z = __uint_as_float(nv.z) - __uint_as_float(ov.z);
            dn.w = __uint_as_float(nv.w) - __uint_as_float(ov.w);
            *reinterpret_cast<f4v*>(drow + sub * 16) = dn;
        }
        *reinterpret_cast<uint4*>(xrow) = nv;
        if (sub == 0) a.stamp0[p] = a.epoch;
    }
    if (SPARSE && tog && sub == 0) memb_spread(a.memb, p, a.next.Hin, a.next.Win, vanish ? -1 : 1, a.epoch);
    // |A_0|: one counter per shard, no returned value to wait for
    const int changed = (int)__popcll(__ballot(gd && sub == 0));
    if (lane == 0 && changed) atomicAdd(a.count0 + shard * CSTRIDE, changed);
    prop_finish<G>(a.next, a.epoch, shard, pb);
}

// Row i of the new list (present pass), valid while i < iend.  ORDER: the
// list must increase strictly (the one-launch form for sorted lists); a row
// not above its predecessor is an input fault.
template <int ROWB, bool BF16, bool SPARSE, bool ORDER>
__device__ __forceinline__ void present_rows(const DetectArgs& a, int i, int iend, int shard) {
    constexpr int G = ROWB / 16;
    const int sub = lane_id() % G;
    bool act = i < iend;
    int p = -1;
    if (act) {
        p = a.idx ? a.idx[i] : i;
        if (p < 0 || p >= a.HW) {
            if (sub == 0) flag_error(a.err, ERR_INDEX_RANGE);
            act = false;
        }
    }
    if constexpr (ORDER) {
        // the next row's cell, from a clamped position, in the same round trip
        const int nx = a.idx[min(i + 1, a.count - 1)];
        if (act && sub == 0 && i + 1 < a.count && nx <= p) flag_error(a.err, nx == p ? ERR_DUPLICATE : ERR_UNSORTED);
    }
    // presence: a pillar marks its cell present for this stride (plain
    // store; the vanish pass checks ownership).  The canvas and feature rows
    // are fetched in the same round trip as the presence word.  Loads are
    // unconditional from clamped addresses (selected afterwards): a load
    // inside a divergent branch makes the compiler drain all outstanding
    // loads where the branch ends.
    const int pc = act ? p : 0;
    const uint64_t mine = ((uint64_t)a.epoch << 32) | (uint32_t)i;
    // sparse backbones: the pillar set itself is an input; a pillar whose
    // cell had none in the previous stride appeared (the word was written by
    // an earlier stride, or never)
    uint64_t op = 0ull;
    if (SPARSE) op = a.pres[pc];
    if (act && sub == 0) a.pres[p] = mine;
    const uint4 ov = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.X) + (size_t)pc * ROWB + sub * 16);
    const uint4 nv = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.feats) +
                                                     (size_t)min(i, a.count - 1) * ROWB + sub * 16);
    const bool tog = SPARSE && act && (op == 0ull || (uint32_t)(op >> 32) != a.epoch - 1u);
    if (a.prev_out && sub == 0 && i < iend) a.prev_out[i] = act ? p : -1;
    emit_rows<ROWB, BF16, SPARSE>(a, p, pc, act, tog, nv, ov, shard, false);
}

// A cell p known to have lost its pillar (valid when act): its old row
// against zero.
template <int ROWB, bool BF16, bool SPARSE>
__device__ __forceinline__ void vanished_rows(const DetectArgs& a, int p, bool act, int shard) {
    constexpr int G = ROWB / 16;
    const int sub = lane_id() % G;
    const int pc = act ? p : 0;
    uint4 ov = make_uint4(0u, 0u, 0u, 0u);
    // a wavefront without a vanished cell skips the load (a uniform branch)
    if (__ballot(act) != 0ull)
        ov = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.X) + (size_t)pc * ROWB + sub * 16);
    emit_rows<ROWB, BF16, SPARSE>(a, p, pc, act, SPARSE && act, make_uint4(0u, 0u, 0u, 0u), ov, shard, true);
}

template <int ROWB, bool BF16, bool VANISH, bool SPARSE>
__global__ __launch_bounds__(256) void detect_kernel(DetectArgs a) {
    constexpr int G = ROWB / 16;   // lanes per feature row
    constexpr int PPW = 64 / G;    // rows per wavefront pass
    const int shard = (int)(blockIdx.x % NSHARD);
    const int lane = lane_id();
    const int sub = lane % G;

    if (!VANISH && a.zero_ptr && blockIdx.x == 0)
        for (int i = threadIdx.x; i < a.zero_n; i += blockDim.x) a.zero_ptr[i] = 0;

    const int wave = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    const int nwaves = (int)((gridDim.x * blockDim.x) >> 6);
    const int rows = VANISH ? max(a.count, a.chk_count) : a.count;
    for (int base = wave * PPW; base < rows; base += nwaves * PPW) {
        const int i = base + lane / G;
        if constexpr (!VANISH) {
            present_rows<ROWB, BF16, SPARSE, false>(a, i, a.count, shard);
        } else {
            bool act = i < a.count;
            int p = -1;
            if (act) {
                p = a.prev ? a.prev[i] : i;
                if (p < 0 || p >= a.HW) act = false;
            }
            const int pc = act ? p : 0;
            const uint64_t mine = ((uint64_t)a.epoch << 32) | (uint32_t)i;
            int c = 0;   // cell of row i of the new list, and its presence word
            if (a.chk_idx) c = a.chk_idx[min(i, a.chk_count - 1)];
            const uint32_t st = (uint32_t)(a.pres[pc] >> 32);
            const uint64_t cw = a.pres[(c >= 0 && c < a.HW) ? c : 0];
            act = act && st != a.epoch;                 // present in this stride: not vanished
            // every pillar of the new list must own its cell's presence word
            // (out-of-range cells were flagged by the present pass)
            if (a.chk_idx && sub == 0 && i < a.chk_count && c >= 0 && c < a.HW && cw != mine)
                flag_error(a.err, ERR_DUPLICATE);
            vanished_rows<ROWB, BF16, SPARSE>(a, p, act, shard);
        }
    }
}

// Sorted pillar lists (cells strictly increasing, the row-major order of a
// pillar scatter): both passes in one launch.  Chunk k of the new list (CH
// rows) owns the cells [lo, hi) from its first row's cell (0 for the first
// chunk) up to the next chunk's first cell (the grid's end for the last), so
// the new pillars in that range are exactly the chunk's rows and a cell of
// the previous list in the range vanished iff it is not one of them: the
// comparison of the two lists stays inside the workgroup.  Wavefronts 0..2
// take the chunk's rows (the present pass); wavefront 3 finds the previous
// list's cells in [lo, hi) by a 32-way sampled search of that sorted list
// (lanes 0-31 for lo, 32-63 for hi, a factor 32 per round trip), tests each
// against the chunk's cells (held one per lane) and processes the vanished
// ones.
template <int ROWB, bool BF16, bool SPARSE>
__global__ __launch_bounds__(256) void detect_sorted_kernel(DetectArgs a) {
    constexpr int G = ROWB / 16;
    constexpr int PPW = 64 / G;
    constexpr int CH = 3 * PPW < 64 ? 3 * PPW : 64;   // rows of a chunk, at most one per lane of wavefront 3
    __shared__ int vq[64];                            // wavefront 3: the vanished cells of a batch
    const int lane = lane_id();
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int shard = (int)(blockIdx.x % NSHARD);
    const int n = a.count, m = a.prev_count;
    const int nchunk = max(1, (n + CH - 1) / CH);

    if (a.zero_ptr && blockIdx.x == 0)
        for (int i = threadIdx.x; i < a.zero_n; i += blockDim.x) a.zero_ptr[i] = 0;

    for (int k = (int)blockIdx.x; k < nchunk; k += (int)gridDim.x) {
        const int i0 = k * CH, i1 = min(i0 + CH, n);
        if (w < 3) {
            if (n > 0 && w * PPW < CH) present_rows<ROWB, BF16, SPARSE, true>(a, i0 + w * PPW + lane / G, i1, shard);
            continue;
        }
        // the chunk's cell range and its cells, one per lane
        const int lo = i0 > 0 ? a.idx[i0] : 0;
        const int hi = i1 < n ? a.idx[i1] : a.HW;
        const int nc = i1 - i0;
        const int cv = n > 0 ? a.idx[min(i0 + lane, n - 1)] : 0;
        // lower bounds of lo (lanes 0-31) and hi (lanes 32-63) in the previous
        // list: the answer stays in [L, R], the entries [L, R) unchecked
        const int x = lane < 32 ? lo : hi;
        const unsigned long long half = lane < 32 ? 0x00000000FFFFFFFFull : 0xFFFFFFFF00000000ull;
        const int sl = lane & 31;
        int L = 0, R = m;
        while (__ballot(L < R) != 0ull) {
            const int len = R - L;
            const int step = (len + 31) / 32;
            const int q = L + (sl + 1) * step - 1;       // sample sl: the last entry of its stretch
            const bool valid = len > 0 && q < R;
            const int v = a.prev[min(max(q, 0), m - 1)];
            const int c = (int)__popcll(__ballot(valid && v < x) & half);   // samples below x: a prefix
            if (len > 0) {
                const int qc = L + (c + 1) * step - 1;   // the first sample not below x, if any
                if (qc < R) R = qc;
                L = L + c * step;
            }
        }
        const int plo = __shfl(L, 0), phi = __shfl(L, 32);
        for (int j0 = plo; j0 < phi; j0 += 64) {
            const int j = j0 + lane;
            const bool in = j < phi;
            const int p = a.prev[min(j, m - 1)];
            // entries of the chunk below p (binary lifting over lanes 0 .. nc-1).
            // Every shuffle runs on the whole wavefront, outside any condition:
            // a lane reading an inactive lane's value gets 0.
            int pos = 0;
#pragma unroll
            for (int b = 32; b >= 1; b >>= 1) {
                const int v = __shfl(cv, min(pos + b - 1, 63));
                if (pos + b <= nc && v < p) pos += b;
            }
            const int at = __shfl(cv, min(pos, 63));
            const bool member = pos < nc && at == p;
            const bool van = in && p >= 0 && p < a.HW && !member;
            const unsigned long long vm = __ballot(van);
            if (van) vq[__popcll(vm & ((1ull << lane) - 1ull))] = p;
            const int nv = (int)__popcll(vm);
            for (int r0 = 0; r0 < nv; r0 += PPW) {
                const int r = r0 + lane / G;
                const bool act = r < nv;
                vanished_rows<ROWB, BF16, SPARSE>(a, vq[act ? r : 0], act, shard);
            }
        }
    }
}

template <bool VANISH>
static hipError_t launch_detect(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    const int G = row_bytes / 16;
    const int ppw = 64 / G;
    const int rows = VANISH ? std::max(a.count, a.chk_count) : a.count;
    long long waves = ((long long)rows + ppw - 1) / ppw;
    long long blocks = (waves + 3) / 4;
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    dim3 grid((unsigned)blocks), block(256);
    const bool sp = a.memb.memb != nullptr;
#define SSC_DETECT_CASE(RB)                                                                             \
    case RB:                                                                                            \
        if (sp)                                                                                         \
            return bf16 ? launch_kernel(c, detect_kernel<RB, true, VANISH, true>, grid, block, a)       \
                        : launch_kernel(c, detect_kernel<RB, false, VANISH, true>, grid, block, a);     \
        return bf16 ? launch_kernel(c, detect_kernel<RB, true, VANISH, false>, grid, block, a)          \
                    : launch_kernel(c, detect_kernel<RB, false, VANISH, false>, grid, block, a);
    switch (row_bytes) {
        SSC_DETECT_CASE(16)
        SSC_DETECT_CASE(32)
        SSC_DETECT_CASE(64)
        SSC_DETECT_CASE(128)
        SSC_DETECT_CASE(256)
        SSC_DETECT_CASE(512)
        SSC_DETECT_CASE(1024)
        default:
            return hipErrorInvalidValue;
    }
#undef SSC_DETECT_CASE
}

hipError_t launch_detect_sorted(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    const int G = row_bytes / 16;
    const int ch = std::min(3 * (64 / G), 64);
    long long blocks = ((long long)a.count + ch - 1) / ch;
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    dim3 grid((unsigned)blocks), block(256);
    const bool sp = a.memb.memb != nullptr;
#define SSC_DETECT_CASE(RB)                                                                          \
    case RB:                                                                                         \
        if (sp)                                                                                      \
            return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, true>, grid, block, a)     \
                        : launch_kernel(c, detect_sorted_kernel<RB, false, true>, grid, block, a);   \
        return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, false>, grid, block, a)        \
                    : launch_kernel(c, detect_sorted_kernel<RB, false, false>, grid, block, a);
    switch (row_bytes) {
        SSC_DETECT_CASE(16)
        SSC_DETECT_CASE(32)
        SSC_DETECT_CASE(64)
        SSC_DETECT_CASE(128)
        SSC_DETECT_CASE(256)
        SSC_DETECT_CASE(512)
        SSC_DETECT_CASE(1024)
        default:
            return hipErrorInvalidValue;
    }
#undef SSC_DETECT_CASE
}

hipError_t launch_detect_present(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    return launch_detect<false>(a, row_bytes, bf16, c);
}

hipError_t launch_detect_vanished(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    return launch_detect<true>(a, row_bytes, bf16, c);
}

}  // namespace ssc
