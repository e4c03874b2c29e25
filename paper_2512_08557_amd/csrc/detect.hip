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
// a separate launch.
// Sparse backbones (SPARSE): the pillar set is itself an input, so a pillar
// that appeared or vanished is changed whatever its values, and it moves the
// first layer's active-set counts (memb_spread).
//
// Layout: G = row_bytes / 16 lanes share one feature row, each lane moving 16
// bytes, so a 64-channel fp32 row (256 B) is one fully coalesced 16-lane
// access.  Delta rows (4*C0 bytes at the cell's position): fp32 new - old, or
// for bf16 the pair [new | old] that the layer kernels contract with
// [W | -W] (exact products, no delta rounding).
#include "device_common.h"

#include <algorithm>

namespace ssc {

template <int ROWB, bool BF16, bool VANISH, bool SPARSE>
__global__ __launch_bounds__(256) void detect_kernel(DetectArgs a) {
    constexpr int G = ROWB / 16;   // lanes per feature row
    constexpr int PPW = 64 / G;    // rows per wavefront pass
    constexpr int DROWB = BF16 ? 2 * ROWB : ROWB;   // delta row bytes
    const int shard = (int)(blockIdx.x % NSHARD);
    const int lane = lane_id();
    const int sub = lane % G;
    const int gbase = lane - sub;

    if (!VANISH && a.zero_ptr && blockIdx.x == 0)
        for (int i = threadIdx.x; i < a.zero_n; i += blockDim.x) a.zero_ptr[i] = 0;

    const int wave = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    const int nwaves = (int)((gridDim.x * blockDim.x) >> 6);
    const int rows = VANISH ? max(a.count, a.chk_count) : a.count;
    for (int base = wave * PPW; base < rows; base += nwaves * PPW) {
        const int i = base + lane / G;
        bool act = i < a.count;
        int p = -1;
        if (act) {
            if (VANISH) p = a.prev ? a.prev[i] : i;
            else p = a.idx ? a.idx[i] : i;
            if (p < 0 || p >= a.HW) {
                if (!VANISH && sub == 0) flag_error(a.err, ERR_INDEX_RANGE);
                act = false;
            }
        }
        // presence: a pillar marks its cell present for this stride (plain
        // store; the vanish pass checks ownership).  The present pass fetches
        // the canvas and feature rows in the same round trip as the presence
        // word; the vanish pass reads a canvas row only after the presence
        // word showed the cell vanished.
        // Loads are unconditional from clamped addresses (selected afterwards):
        // a load inside a divergent branch makes the compiler drain all
        // outstanding loads where the branch ends.
        const int pc = act ? p : 0;
        const uint64_t mine = ((uint64_t)a.epoch << 32) | (uint32_t)i;
        // sparse backbones: the pillar set itself is an input; a pillar whose
        // cell had none in the previous stride appeared (the word was
        // written by an earlier stride, or never)
        uint64_t op = 0ull;
        if (SPARSE && !VANISH) op = a.pres[pc];
        uint32_t st = 0u;
        int c = 0;              // vanish mode: cell of row i of the new list
        uint64_t cw = 0ull;     // and its presence word
        if (VANISH) {
            if (a.chk_idx) c = a.chk_idx[min(i, a.chk_count - 1)];
            st = (uint32_t)(a.pres[pc] >> 32);
            cw = a.pres[(c >= 0 && c < a.HW) ? c : 0];
        } else if (act && sub == 0) {
            a.pres[p] = mine;
        }
        char* xrow = static_cast<char*>(a.X) + (size_t)pc * ROWB + sub * 16;
        uint4 ov = make_uint4(0u, 0u, 0u, 0u);
        uint4 nv = make_uint4(0u, 0u, 0u, 0u);
        if (!VANISH) {
            ov = *reinterpret_cast<const uint4*>(xrow);
            nv = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.feats) +
                                                 (size_t)min(i, a.count - 1) * ROWB + sub * 16);
        } else {
            act = act && st != a.epoch;                 // present in this stride: not vanished
            // every pillar of the new list must own its cell's presence word
            // (out-of-range cells were flagged by the present pass)
            if (a.chk_idx && sub == 0 && i < a.chk_count && c >= 0 && c < a.HW && cw != mine)
                flag_error(a.err, ERR_DUPLICATE);
            // only the canvas rows of vanished cells are read: most cells of
            // the previous list are present again, and a wavefront without a
            // vanished cell skips the load (a uniform branch)
            if (__ballot(act) != 0ull) ov = *reinterpret_cast<const uint4*>(xrow);
        }
        bool tog = false;       // sparse backbones: the pillar appeared or vanished
        if (SPARSE) tog = VANISH ? act : (act && (op == 0ull || (uint32_t)(op >> 32) != a.epoch - 1u));
        const bool d = act && (tog || nv.x != ov.x || nv.y != ov.y || nv.z != ov.z || nv.w != ov.w);
        const unsigned long long bal = __ballot(d);
        const unsigned long long gm = (G == 64 ? ~0ull : ((1ull << G) - 1ull)) << gbase;
        const bool gd = (bal & gm) != 0ull;
        // stamp the first layer's footprint while the rows are written
        PropBatch<G> pb;
        prop_issue<G, false>(a.next, pc, gd, sub, a.epoch, pb);
        if (gd) {
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
        if (SPARSE && tog && sub == 0) memb_spread(a.memb, p, a.next.Hin, a.next.Win, VANISH ? -1 : 1, a.epoch);
        // |A_0|: one counter per shard, no returned value to wait for
        const int changed = (int)__popcll(__ballot(gd && sub == 0));
        if (lane == 0 && changed) atomicAdd(a.count0 + shard * CSTRIDE, changed);
        if (!VANISH && a.prev_out && sub == 0 && i < a.count) a.prev_out[i] = act ? p : -1;
        prop_finish<G>(a.next, a.epoch, shard, pb);
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

hipError_t launch_detect_present(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    return launch_detect<false>(a, row_bytes, bf16, c);
}

hipError_t launch_detect_vanished(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
    return launch_detect<true>(a, row_bytes, bf16, c);
}

}  // namespace ssc
