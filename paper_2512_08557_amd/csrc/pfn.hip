// Incremental pillar feature net: the point-level front end of a stride
// (Sec. III-B; Alg. 1, PFN part).
//
// Per stride, two launches replace change detection on feature rows:
//   pillar_update : the points of the stride that leaves the window are
//                   removed from their pillars' queues and the new stride's
//                   points are inserted; every pillar that loses or gains a
//                   point is changed (the event-based change map of Alg. 1)
//                   and goes to the A_0 list;
//   pfn           : for each changed pillar, its window's points are decorated
//                   (x, y, z, intensity, offsets from the pillar centre,
//                   offsets from the points' mean: D = 9), mapped by the
//                   pointwise linear layer (batch norm folded, no bias), ReLU,
//                   and max-pooled over the points into the pillar's C0
//                   features; a pillar without points is empty (zero row).
//                   The canvas, the input deltas and the A_0 -> A_1
//                   propagation follow, exactly as change detection does them.
// A pillar holds at most N points (the paper's N = 100); more is an input
// fault (ERR_PILLAR_FULL), never sampling.
//
// Binning decides an integer from floating point: column = floor((x - x_min)
// * inv_res) with every operation rounded to float32 and inv_res = 1/res
// rounded to float32; a point is in the grid when 0 <= that < W (and the same
// for rows), so NaN coordinates fall outside.
#include "device_common.h"

#include <algorithm>

namespace ssc {

// Appends `value` of every lane with `mine` set to the list `seg` with
// counter `cnt`, one atomic per wavefront.  Every active lane must call it.
__device__ __forceinline__ void wave_append(int32_t* cnt, int32_t* seg, bool mine, int32_t value) {
    const unsigned long long m = __ballot(mine);
    if (m == 0ull) return;
    const int lane = lane_id();
    const int first = __ffsll((long long)m) - 1;
    int base = 0;
    if (lane == first) base = atomicAdd(cnt, (int)__popcll(m));
    base = __shfl(base, first);
    if (mine) seg[base + (int)__popcll(m & ((1ull << lane) - 1ull))] = value;
}

// wave_append to two lists at once: both counters' atomics are issued before
// either result is waited for.
__device__ __forceinline__ void wave_append2(int32_t* cnt_a, int32_t* seg_a, bool mine_a,
                                             int32_t* cnt_b, int32_t* seg_b, bool mine_b, int32_t value) {
    const unsigned long long ma = __ballot(mine_a), mb = __ballot(mine_b);
    if ((ma | mb) == 0ull) return;
    const int lane = lane_id();
    const int fa = ma ? __ffsll((long long)ma) - 1 : 0, fb = mb ? __ffsll((long long)mb) - 1 : 0;
    int ba = 0, bb = 0;
    if (ma && lane == fa) ba = atomicAdd(cnt_a, (int)__popcll(ma));
    if (mb && lane == fb) bb = atomicAdd(cnt_b, (int)__popcll(mb));
    ba = __shfl(ba, fa);
    bb = __shfl(bb, fb);
    const unsigned long long below = (1ull << lane) - 1ull;
    if (mine_a) seg_a[ba + (int)__popcll(ma & below)] = value;
    if (mine_b) seg_b[bb + (int)__popcll(mb & below)] = value;
}

__global__ __launch_bounds__(256) void pillar_update_kernel(PillarArgs a) {
    const int lane = lane_id(), wave = (int)(threadIdx.x >> 6);
    const int shard = (int)(blockIdx.x % NSHARD);
    int32_t* cnt0 = a.count0 + shard * CSTRIDE;
    int32_t* seg0 = a.list0 + (size_t)shard * ((size_t)a.H * a.W);
    if (a.zero_ptr && blockIdx.x == 0)
        for (int i = (int)threadIdx.x; i < a.zero_n; i += (int)blockDim.x) a.zero_ptr[(size_t)i * CSTRIDE] = 0;

    if ((int)blockIdx.x < a.n_pop_blocks) {
        // the stride leaving the window: its cells are unique in its list
        const int n = *a.tcount_pop;
        for (int base = (int)blockIdx.x * 256 + wave * 64; base < n; base += a.n_pop_blocks * 256) {
            const int i = base + lane;
            const bool v = i < n;
            const int c = v ? a.touched_pop[i] : 0;
            bool first = false;
            if (v) {
                // both loads and the stamp in one round trip
                const uint32_t k = a.scnt_pop[c];
                const uint32_t h = a.head[c];
                const uint32_t old = atomicMax(&a.stamp0[c], a.epoch);
                a.scnt_pop[c] = 0u;
                a.head[c] = h + k;
                first = old < a.epoch;
            }
            wave_append(cnt0, seg0, first, c);
        }
    } else {
        const int b = (int)blockIdx.x - a.n_pop_blocks;
        const int nb = (int)gridDim.x - a.n_pop_blocks;
        for (int base = b * 256 + wave * 64; base < a.n_points; base += nb * 256) {
            const int i = base + lane;
            bool v = i < a.n_points;
            const float4 p = a.points[v ? i : 0];
            const float fx = __fmul_rn(__fsub_rn(p.x, a.x_min), a.inv_res);
            const float fy = __fmul_rn(__fsub_rn(p.y, a.y_min), a.inv_res);
            v = v && fx >= 0.f && fx < (float)a.W && fy >= 0.f && fy < (float)a.H;
            const int c = v ? (int)fy * a.W + (int)fx : 0;
            bool first_ins = false, first_chg = false;
            if (v) {
                // the four atomics in one round trip, the ring store after
                const uint32_t pos = atomicAdd(&a.tail[c], 1u);
                atomicAdd(&a.scnt_ins[c], 1u);
                const uint32_t oi = atomicMax(&a.ins_stamp[c], a.epoch);
                const uint32_t oc = atomicMax(&a.stamp0[c], a.epoch);
                a.ring[(size_t)c * a.N + pos % (uint32_t)a.N] = p;
                first_ins = oi < a.epoch;
                first_chg = oc < a.epoch;
            }
            wave_append2(a.tcount_ins, a.touched_ins, first_ins, cnt0, seg0, first_chg, c);
        }
    }
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ __forceinline__ float bcast(float v, int src) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), src));
}

// One wavefront per changed pillar; lane k computes output channel k.  The
// pillar's points sit one per lane (two per lane beyond 64), their decoration
// is broadcast point by point.  The point sums use float64: coordinates below
// 2^6 m in float32 and at most 128 terms stay exact in its 53 bits, so the
// mean does not depend on the order the points were inserted in.
template <bool BF16>
__global__ __launch_bounds__(256) void pfn_kernel(PfnArgs a) {
    const int lane = lane_id(), wave = (int)(threadIdx.x >> 6);
    const int shard = (int)(blockIdx.x % NSHARD);
    if (blockIdx.x == 0 && threadIdx.x == 0) *a.tcount_clear = 0;
    int cnt[NSHARD];
    int total = 0;
#pragma unroll
    for (int k = 0; k < NSHARD; ++k) {
        cnt[k] = a.count0[k * CSTRIDE];
        total += cnt[k];
    }
    float wk[9];
#pragma unroll
    for (int d = 0; d < 9; ++d) wk[d] = lane < a.C0 ? a.w[lane * 9 + d] : 0.f;

    for (int g = (int)blockIdx.x * 4 + wave; g < total; g += (int)gridDim.x * 4) {
        int k = 0, gi = g;
#pragma unroll
        for (int s = 0; s < NSHARD - 1; ++s)
            if (k == s && gi >= cnt[s]) {
                gi -= cnt[s];
                k = s + 1;
            }
        const int c = a.list0[(size_t)k * a.cap0 + gi];
        // the queue bounds, the old canvas value of this lane's channel and
        // the next layer's footprint stamps in one round trip (none depends
        // on the new features: the pillar changed because its points did)
        const uint32_t hd = a.head[c];
        const uint32_t tl = a.tail[c];
        const int ch = lane < a.C0 ? lane : 0;
        float xo_f = 0.f;
        uint16_t xo_b = 0;
        if constexpr (BF16) xo_b = static_cast<const uint16_t*>(a.X)[(size_t)c * a.C0 + ch];
        else xo_f = static_cast<const float*>(a.X)[(size_t)c * a.C0 + ch];
        PropBatch<64> pb;
        prop_issue<64, false>(a.next, c, true, lane, a.epoch, pb);
        int n = (int)(tl - hd);
        if (n > a.N) {
            if (lane == 0) flag_error(a.err, ERR_PILLAR_FULL);
            n = a.N;
        }
        const float4* rq = a.ring + (size_t)c * a.N;
        const bool h0 = lane < n, h1 = lane + 64 < n;
        const float4 z4 = make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 p0 = h0 ? rq[(hd + (uint32_t)lane) % (uint32_t)a.N] : z4;
        const float4 p1 = h1 ? rq[(hd + (uint32_t)lane + 64u) % (uint32_t)a.N] : z4;
        // the list positions, while the points arrive: the counter's round
        // trip overlaps them and the feature computation
        PropSlots<64> ps;
        prop_reserve<64>(a.next, a.epoch, shard, pb, ps);
        const double sx = wave_sum((double)p0.x + (double)p1.x);
        const double sy = wave_sum((double)p0.y + (double)p1.y);
        const double sz = wave_sum((double)p0.z + (double)p1.z);
        const double inv_n = n > 0 ? 1.0 / n : 0.0;
        const float mx = (float)(sx * inv_n), my = (float)(sy * inv_n), mz = (float)(sz * inv_n);
        const int row = c / a.W, col = c - (c / a.W) * a.W;
        const float cx = a.x_min + ((float)col + 0.5f) * a.res;
        const float cy = a.y_min + ((float)row + 0.5f) * a.res;
        const float d0[9] = {p0.x, p0.y, p0.z, p0.w, p0.x - cx, p0.y - cy, p0.x - mx, p0.y - my, p0.z - mz};
        const float d1[9] = {p1.x, p1.y, p1.z, p1.w, p1.x - cx, p1.y - cy, p1.x - mx, p1.y - my, p1.z - mz};
        float f = 0.f;                           // max over points of ReLU(w . d)
        for (int j = 0; j < n; ++j) {
            const int src = j & 63;
            float v = 0.f;
            if (j < 64) {
#pragma unroll
                for (int d = 0; d < 9; ++d) v = fmaf(wk[d], bcast(d0[d], src), v);
            } else {
#pragma unroll
                for (int d = 0; d < 9; ++d) v = fmaf(wk[d], bcast(d1[d], src), v);
            }
            f = fmaxf(f, v);
        }

        if (lane < a.C0) {
            if constexpr (BF16) {
                uint16_t* x = static_cast<uint16_t*>(a.X) + (size_t)c * a.C0 + lane;
                uint16_t* dr = static_cast<uint16_t*>(a.delta0) + (size_t)c * 2 * a.C0;
                const uint16_t nb = (uint16_t)f32_to_bf16_bits(f);
                dr[lane] = nb;                   // the pair [new | old]
                dr[a.C0 + lane] = xo_b;
                *x = nb;
            } else {
                float* x = static_cast<float*>(a.X) + (size_t)c * a.C0 + lane;
                static_cast<float*>(a.delta0)[(size_t)c * a.C0 + lane] = f - xo_f;
                *x = f;
            }
        }
        prop_write<64>(a.next, shard, pb, ps);
    }
}

hipError_t launch_pillar_update(const PillarArgs& a, int insert_blocks, const LaunchCtx& c) {
    return launch_kernel(c, pillar_update_kernel, dim3(a.n_pop_blocks + std::max(insert_blocks, 1)), dim3(256), a);
}

hipError_t launch_pfn(const PfnArgs& a, bool bf16, int blocks, const LaunchCtx& c) {
    return bf16 ? launch_kernel(c, pfn_kernel<true>, dim3(blocks), dim3(256), a)
                : launch_kernel(c, pfn_kernel<false>, dim3(blocks), dim3(256), a);
}

}  // namespace ssc
