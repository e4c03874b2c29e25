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
// first layer's active-set counts (memb_issue, memb_swap, memb_settle).
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
    // stamp the first layer's footprint while the rows are written; a
    // toggled pillar's active-set targets load in the same round trip
    PropBatch<G> pb;
    prop_issue<G, false>(a.next, pc, gd, sub, a.epoch, pb);
    MembBatch mb;
    const int md = vanish ? -1 : 1;
    // (only a wavefront with a toggle loads them: the branch is uniform)
    const bool mtog = SPARSE && __ballot(tog && sub == 0) != 0ull;
    if (mtog) memb_issue(a.memb, pc, a.next.Hin, a.next.Win, tog && sub == 0, mb);
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
    // the swaps' round trip overlaps the list append's
    unsigned long long got[9];
    if (mtog) memb_swap(a.memb, pc, a.next.Hin, a.next.Win, mb, md, a.epoch, got);
    // |A_0|: one counter per shard, no returned value to wait for
    const int changed = (int)__popcll(__ballot(gd && sub == 0));
    if (lane == 0 && changed)
        atomicAdd(a.count0 + (shard * PSPREAD + (int)(blockIdx.x & (PSPREAD - 1))) * CSTRIDE, changed);
    prop_finish<G>(a.next, a.epoch, shard, pb);
    if (mtog) memb_settle(a.memb, pc, a.next.Hin, a.next.Win, mb, md, a.epoch, got);
}

// Rows i + u*step (u < U) of the new list (present pass), each valid while
// below iend; a.count >= 1.  Every row's cell is loaded first, then every
// row's canvas and feature pieces, so all U rows' loads are in flight
// together before the first comparison.  a.sorted: the list was passed as
// increasing strictly; a row not above its predecessor is an input fault.
template <int ROWB, bool BF16, bool SPARSE, int U>
__device__ __forceinline__ void present_rows(const DetectArgs& a, int i, int step, int iend, int shard) {
    constexpr int G = ROWB / 16;
    const int sub = lane_id() % G;
    // loads are unconditional from clamped addresses (selected afterwards):
    // a load inside a divergent branch makes the compiler drain all
    // outstanding loads where the branch ends
    int p[U], nx[U];
    bool act[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = i + u * step;
        act[u] = r < iend;
        p[u] = a.idx ? a.idx[min(r, a.count - 1)] : r;
        // the next row's cell, for the order check, in the same round trip
        nx[u] = a.sorted ? a.idx[min(r + 1, a.count - 1)] : 0;
    }
    int pc[U];
    uint64_t op[U];
    uint4 ov[U], nv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = i + u * step;
        if (act[u] && (p[u] < 0 || p[u] >= a.HW)) {
            if (sub == 0) flag_error(a.err, ERR_INDEX_RANGE);
            act[u] = false;
        }
        if (a.sorted && act[u] && sub == 0 && r + 1 < a.count && nx[u] <= p[u])
            flag_error(a.err, nx[u] == p[u] ? ERR_DUPLICATE : ERR_UNSORTED);
        // presence: a pillar marks its cell present for this stride (plain
        // store; the vanish pass checks ownership).  The canvas and feature
        // rows are fetched in the same round trip as the presence word.
        pc[u] = act[u] ? p[u] : 0;
        // sparse backbones: the pillar set itself is an input; a pillar
        // whose cell had none in the previous stride appeared (the word was
        // written by an earlier stride, or never)
        op[u] = SPARSE ? a.pres[pc[u]] : 0ull;
        if (act[u] && sub == 0) a.pres[p[u]] = ((uint64_t)a.epoch << 32) | (uint32_t)r;
        ov[u] = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.X) + (size_t)pc[u] * ROWB + sub * 16);
        nv[u] = *reinterpret_cast<const uint4*>(static_cast<const char*>(a.feats) +
                                                (size_t)min(r, a.count - 1) * ROWB + sub * 16);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int r = i + u * step;
        const bool tog = SPARSE && act[u] && (op[u] == 0ull || (uint32_t)(op[u] >> 32) != a.epoch - 1u);
        if (a.prev_out && sub == 0 && r < iend) a.prev_out[r] = act[u] ? p[u] : -1;
        emit_rows<ROWB, BF16, SPARSE>(a, p[u], pc[u], act[u], tog, nv[u], ov[u], shard, false);
    }
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
        for (int i = threadIdx.x; i < a.zero_n; i += blockDim.x) a.zero_ptr[(size_t)i * CSTRIDE] = 0;

    const int wave = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    const int nwaves = (int)((gridDim.x * blockDim.x) >> 6);
    const int rows = VANISH ? max(a.count, a.chk_count) : a.count;
    for (int base = wave * PPW; base < rows; base += nwaves * PPW) {
        const int i = base + lane / G;
        if constexpr (!VANISH) {
            present_rows<ROWB, BF16, SPARSE, 1>(a, i, 0, a.count, shard);
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

// Lower bound of x in the sorted list v[0, len) (the first position whose
// cell is not below x), computed by the 32 lanes of one half-wavefront
// together: each round loads 32 evenly spaced samples of the remaining
// stretch and keeps the stretch between the last sample below x and the
// first one not below it, a factor 32 per round trip.  `half` masks this
// half's lanes; both halves run the same rounds (a uniform loop), each with
// its own x.
__device__ __forceinline__ int lower_bound32(const int32_t* __restrict__ v, int len, int x,
                                             unsigned long long half) {
    const int sl = lane_id() & 31;
    int L = 0, R = len;        // the answer is in [L, R]; entries [L, R) unchecked
    while (__ballot(L < R) != 0ull) {
        const int n = R - L;
        const int step = (n + 31) / 32;
        const int q = L + (sl + 1) * step - 1;      // sample sl: the last entry of its stretch
        const bool valid = n > 0 && q < R;
        const int s = v[min(max(q, 0), max(len - 1, 0))];
        const int c = (int)__popcll(__ballot(valid && s < x) & half);   // samples below x: a prefix
        if (n > 0) {
            const int qc = L + (c + 1) * step - 1;  // the first sample not below x, if any
            if (qc < R) R = qc;
            L = L + c * step;
        }
    }
    return L;
}

// Rows of the new list per workgroup of the sorted detection: the three
// present wavefronts take U passes of PPW rows each (at most 64 rows, the
// size of the previous-list chunk).  U = 1 while one pass per workgroup puts
// the whole list into one round of resident workgroups; a longer list takes
// UB passes, all their loads in flight together, so that it needs fewer
// rounds of the chunk's dependent round trips (four 1024x1024 images: ~13k
// chunks of 12 rows otherwise).
template <int ROWB>
struct SortedChunk {
    static constexpr int PPW = 64 / (ROWB / 16);
    static constexpr int UB = 3 * PPW >= 64 ? 1 : (64 / (3 * PPW) < 8 ? 64 / (3 * PPW) : 8);
    static constexpr int rows(int u) { return 3 * PPW * u < 64 ? 3 * PPW * u : 64; }
};

// Sorted pillar lists (cells strictly increasing, the row-major order of a
// pillar scatter): both passes in one launch, every comparison of the two
// lists inside one workgroup.  Workgroup k takes rows k*CH .. of the new list
// (the present pass, wavefronts 0..2) and entries 64k .. 64k+63 of the
// previous list (wavefront 3): a previous cell p vanished iff the new list
// does not hold p.  Wavefront 3 finds the stretch of the new list between its
// first and last previous cell by a 32-way sampled search (lanes 0-31 and
// 32-63 for the two ends), then tests each of its cells against that stretch:
// by binary lifting over shuffles when the stretch fits the 64 lanes, else by
// a binary search per lane (a region of new pillars between two previous
// ones).  The vanished cells (at most 64) go to LDS and all four wavefronts
// process them.  Each workgroup's work is bounded by its two chunks, so a
// region that loses all its pillars at once spreads over the workgroups of
// its stretch of the previous list.
// U: rows of the new list per lane group and wavefront (SortedChunk).
template <int ROWB, bool BF16, bool SPARSE, int U>
__global__ __launch_bounds__(256) void detect_sorted_kernel(DetectArgs a) {
    constexpr int G = ROWB / 16;
    constexpr int PPW = 64 / G;
    constexpr int CH = SortedChunk<ROWB>::rows(U);    // rows of the new list per workgroup
    __shared__ int vq[64];                            // the vanished cells of the workgroup's previous chunk
    __shared__ int nvq;
    const int lane = lane_id();
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int shard = (int)(blockIdx.x % NSHARD);
    const int n = a.count, m = a.prev_count;
    const int nchunk = max(max((n + CH - 1) / CH, (m + 63) / 64), 1);

    if (a.zero_ptr && blockIdx.x == 0)
        for (int i = threadIdx.x; i < a.zero_n; i += blockDim.x) a.zero_ptr[(size_t)i * CSTRIDE] = 0;

    for (int k = (int)blockIdx.x; k < nchunk; k += (int)gridDim.x) {
        if (w < 3) {
            const int i0 = k * CH;
            if (i0 < n && w * PPW < CH)
                present_rows<ROWB, BF16, SPARSE, U>(a, i0 + w * PPW + lane / G, 3 * PPW, min(i0 + CH, n), shard);
        } else {
            const int j0 = 64 * k;
            int nv = 0;
            if (j0 < m) {
                const int np = min(64, m - j0);
                const bool in = lane < np;
                const int p = a.prev[j0 + (in ? lane : 0)];
                // the new list's stretch [b0, b1) of cells in [first, last] of
                // this chunk (both ends searched at once)
                const int first = a.prev[j0], last = a.prev[j0 + np - 1];
                const unsigned long long half = lane < 32 ? 0x00000000FFFFFFFFull : 0xFFFFFFFF00000000ull;
                const int L = lower_bound32(a.idx, n, lane < 32 ? first : last + 1, half);
                const int b0 = __shfl(L, 0), b1 = __shfl(L, 32);
                const int len = b1 - b0;
                bool member = false;
                if (len <= 64) {
                    // the stretch one cell per lane; every shuffle runs on the
                    // whole wavefront (a lane reading an inactive lane gets 0)
                    const int cv = len > 0 ? a.idx[b0 + min(lane, len - 1)] : 0;
                    int pos = 0;
#pragma unroll
                    for (int b = 32; b >= 1; b >>= 1) {
                        const int v = __shfl(cv, min(pos + b - 1, 63));
                        if (pos + b <= len && v < p) pos += b;
                    }
                    const int at = __shfl(cv, min(pos, 63));
                    member = pos < len && at == p;
                } else {
                    // a long stretch: binary search per lane in the new list
                    int lo = b0, hi = b1;
                    while (__ballot(lo < hi) != 0ull) {
                        const int mid = (lo + hi) >> 1;
                        const int v = a.idx[min(mid, n - 1)];
                        if (lo < hi) {
                            if (v < p) lo = mid + 1;
                            else hi = mid;
                        }
                    }
                    member = lo < b1 && a.idx[min(lo, n - 1)] == p;
                }
                const bool van = in && p >= 0 && p < a.HW && !member;
                const unsigned long long vm = __ballot(van);
                if (van) vq[__popcll(vm & ((1ull << lane) - 1ull))] = p;
                nv = (int)__popcll(vm);
            }
            if (lane == 0) nvq = nv;
        }
        // the chunk's vanished cells, PPW per wavefront pass over all four
        __syncthreads();
        const int nv = nvq;
        for (int r0 = w * PPW; r0 < nv; r0 += 4 * PPW) {
            const int r = r0 + lane / G;
            const bool act = r < nv;
            vanished_rows<ROWB, BF16, SPARSE>(a, vq[act ? r : 0], act, shard);
        }
        __syncthreads();   // vq and nvq are rewritten by the next chunk
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

// resident workgroups of detect_sorted_kernel (256 threads) on 256 compute units
constexpr long long SORTED_ROUND = 2048;

template <int RB>
static hipError_t launch_ds(const DetectArgs& a, bool bf16, const LaunchCtx& c) {
    using SC = SortedChunk<RB>;
    const bool wide = (long long)a.count > SORTED_ROUND * SC::rows(1);
    const int ch = SC::rows(wide ? SC::UB : 1);
    long long blocks = std::max(((long long)a.count + ch - 1) / ch, ((long long)a.prev_count + 63) / 64);
    if (blocks < 1) blocks = 1;
    if (blocks > 4096) blocks = 4096;
    dim3 grid((unsigned)blocks), block(256);
    const bool sp = a.memb.memb != nullptr;
    if (wide) {
        if (sp) return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, true, SC::UB>, grid, block, a)
                            : launch_kernel(c, detect_sorted_kernel<RB, false, true, SC::UB>, grid, block, a);
        return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, false, SC::UB>, grid, block, a)
                    : launch_kernel(c, detect_sorted_kernel<RB, false, false, SC::UB>, grid, block, a);
    }
    if (sp) return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, true, 1>, grid, block, a)
                        : launch_kernel(c, detect_sorted_kernel<RB, false, true, 1>, grid, block, a);
    return bf16 ? launch_kernel(c, detect_sorted_kernel<RB, true, false, 1>, grid, block, a)
                : launch_kernel(c, detect_sorted_kernel<RB, false, false, 1>, grid, block, a);
}

hipError_t launch_detect_sorted(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c) {
#define SSC_DETECT_CASE(RB) \
    case RB:                \
        return launch_ds<RB>(a, bf16, c);
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
