// One convolution layer of a stride, on the changed cells only.
//
// Method (SSCATeR, arXiv 2512.08557, Eq. 2 and Alg. 1 backbone part): every
// changed input site scatters (I_curr - I_prev) x W[m, n] into the persistent
// output map; the touched output sites form the layer's change list; the next
// layer's input delta at a changed site is phi(Z_new) - phi(Z_old).
//
// Dataflow on gfx950 (output-stationary; no atomics on the maps):
//   * the change list A_l of this layer's OUTPUT grid was built by the
//     previous launch (scatter rule), so every output cell that receives a
//     scatter contribution is known up front;
//   * a workgroup owns 16 consecutive cells of one segment of A_l and all
//     output channels.  For each of the 9 taps it checks the change stamps
//     of the input cells under that tap and gathers the delta rows of the
//     changed ones (stored at their cells; unchanged inputs contribute zero
//     and a tap with no changed input in the whole tile is skipped), then
//     contracts them with the tap's weights on the matrix cores:
//     D[cout x 16 cells] += W_t^T[cout x cin] . dY^T.
//     Summing the 9 taps per output cell in a fixed order is exactly the sum
//     the scatter of Eq. 2 adds into that cell, so the result is
//     deterministic and each Z row is read and written once per stride;
//   * epilogue in registers: Z_new = Z_old + D; store Z_new; write the next
//     layer's delta row at the cell (fp32 phi(Z_new) - phi(Z_old), or the bf16
//     pair [bf16(phi(Z_new)) | bf16(phi(Z_old))]);
//   * wavefront 0 then propagates the tile's cells to the next layer's change
//     list (the structural rule, including stride-2 downsampling).
//
// MFMA operand layout (v_mfma_f32_16x16x4_f32; v_mfma_f32_16x16x32_bf16):
//   src0 = weights, lane l supplies rows cout = l%16 of k-group l/16;
//   src1 = deltas,  lane l supplies cell l%16 of k-group l/16;
//   D: lane l, register j holds cout 4*(l/16)+j of cell l%16.
// With k-group g = l/16 covering 4 (fp32) or 8 (bf16) consecutive k, one
// lane's delta operand for a 16-channel (fp32) or 32-value (bf16 pair) chunk
// is a single contiguous 16-byte load and the weight operand another, both
// fully coalesced; D is four consecutive output channels of one cell, so the Z
// update is a 16-byte load/store per lane.
//
// Workgroup b walks the tiles of list segment (b / 8) % NSHARD; the
// segments are filled by different workgroups of the previous launch so that
// no single counter takes every append.
//
// Sparse backbones (SPARSE = true): a site inactive in this and in the
// previous stride neither changes nor propagates; an inactive site's output is
// zero in the delta epilogue; the first layer of a block passes its sites'
// membership changes to the next block's active-set counts.  Z is updated at
// every site of the list, active or not, so a site that joins the active set
// already holds its sum.
#include "device_common.h"

#include <string.h>

#include <algorithm>

namespace ssc {

// COUT = 8 takes one 16-wide block whose upper 8 weight rows are zero; the
// lanes holding those rows (k-groups 2 and 3) neither read nor write Z.
// NWC wavefronts cover the cout blocks; with a single block (COUT <= 16)
// KS = 4 wavefronts split the contraction (the (tap, chunk) steps) and add
// their partial sums through LDS (measured: a 2-way split at COUT = 32 is
// slower than 2 wavefronts with the whole contraction each).
// A stride-2 layer with more than four blocks (cout 128 and 256) spreads
// them over CS workgroups per tile, one block per wavefront each (four per
// workgroup, two for bf16 and sparse layers), on the same XCD: its output list is ~4x shorter than its input list (the c3/c4 layer
// 64->128: ~80 tiles, fewer than the compute units), so a wavefront's matrix
// work is the chain that ends the launch.  With four blocks (cout 64) the
// tile's two workgroups take two blocks each: twice the compute units, each
// streaming half the tile's operands (block 1's first layer: 68 tiles on
// 432x496, 0.5-1 us shorter per launch).  (Stride 1 with ~170 tiles: the
// split only doubles the gathers; measured 1 us slower per launch.)
// bf16 weights: the pair form contracts [Y_new | Y_old] against [W | -W];
// the packed weights hold W once (chunk c of the pair uses weight chunk
// c % N) and the kernels flip the sign bits of the delta's old half
// instead, which gives bit-identical products ((-y) * w == y * (-w)).  With
// cin = 16 the one 32-value chunk holds [W | W].
template <int CIN, bool BF16>
struct WeightChunks {
    static constexpr int N = BF16 ? (CIN >= 32 ? CIN / 32 : 1) : CIN / 16;
};

// The 8 bf16 pair values of lane group g in chunk c, their sign bits flipped
// where they belong to the old half (pair position >= CIN).
template <int CIN>
__device__ __forceinline__ uint4 old_half_negated(uint4 v, int c, int g) {
    const uint32_t s = c * 32 + 8 * g >= CIN ? 0x80008000u : 0u;
    return make_uint4(v.x ^ s, v.y ^ s, v.z ^ s, v.w ^ s);
}

// FINE: bf16 or sparse layers, whose stride-2 tiles with more than four
// blocks spread over workgroups of two blocks (measured faster there; four
// blocks per workgroup measured faster for dense fp32 layers).
template <int COUT, int S = 1, bool FINE = false>
struct LayerShape {
    static constexpr int NCBT = (COUT + 15) / 16;           // 16-wide cout blocks
    // workgroups per tile (cout parts)
    static constexpr int CS = S == 2 ? (NCBT > 4 ? NCBT / (FINE ? 2 : 4) : (NCBT == 4 ? 2 : 1)) : 1;
    static constexpr int NCBW = NCBT / CS;                  // cout blocks per workgroup
    static constexpr int NWC = NCBW >= 4 ? 4 : NCBW;        // wavefronts across the cout blocks
    static constexpr int KS = NWC == 1 ? 4 : 1;             // wavefronts across the contraction
    static constexpr int NW = NWC * KS;                     // wavefronts per workgroup
    static constexpr int NCB = NCBW / NWC;                  // cout blocks per wavefront
};

// One 16-channel (fp32) or 32-value (bf16 pair) chunk of the contraction for
// NCB output blocks: D[cb] += W_cb^T . dY^T.
template <bool BF16, int NCB>
__device__ __forceinline__ void mfma_chunk(f4v (&acc)[NCB], const uint4 av, const uint4 (&bv)[NCB]) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        if constexpr (BF16) {
            bf8v A, B;
            __builtin_memcpy(&A, &bv[cb], 16);
            __builtin_memcpy(&B, &av, 16);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[cb], 0, 0, 0);
        } else {
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].x), __uint_as_float(av.x), acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].y), __uint_as_float(av.y), acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].z), __uint_as_float(av.z), acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].w), __uint_as_float(av.w), acc[cb], 0, 0, 0);
        }
    }
}

// plist, pcount, pcap are a.list, a.count, a.cap passed again as leading
// scalar arguments: the build preloads them into SGPRs, so the list entry and
// count loads that open every tile need not wait for the argument fetch.
// SPREAD (with SPARSE): the layer is regular and the next regular layer's
// active-set counts follow its sites (a.mnext set).
template <int CIN, int COUT, int S, bool BF16, bool SPARSE, bool SPREAD>
__global__ __launch_bounds__((64 * LayerShape<COUT, S, BF16 || SPARSE>::NW)) void layer_kernel(const int32_t* __restrict__ plist,
                                                                          const int32_t* __restrict__ pcount, int pcap,
                                                                          LayerArgs a) {
    using LS = LayerShape<COUT, S, BF16 || SPARSE>;
    constexpr int NCBT = LS::NCBT;
    constexpr int NCB = LS::NCB;
    constexpr int NWC = LS::NWC, KS = LS::KS;
    constexpr int CS = LS::CS, NCBW = LS::NCBW;
    constexpr int KTOT = BF16 ? 2 * CIN : CIN;   // contraction length per tap
    constexpr int KCH = BF16 ? 32 : 16;          // k per 64-byte chunk
    constexpr int NCH = KTOT / KCH;
    constexpr int NCHW = WeightChunks<CIN, BF16>::N;   // weight chunks per tap
    constexpr int ROWB_IN = 4 * CIN;             // input delta row bytes (fp32, or bf16 pair)

    const int lane = (int)(threadIdx.x & 63u), wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int cl = lane & 15, g = lane >> 4;
    const int cw = wave % NWC, ks = wave / NWC;  // cout group, contraction share
    const int G = (int)gridDim.x;                // a multiple of 32 * NSHARD * CS

    // tiles of segment (b / (8 * CS)) % NSHARD, first one without waiting
    // for the count.  The workgroups of a segment sit on all eight XCDs
    // (workgroup b runs on XCD b % 8), so an uneven split of the list over
    // the segments does not load one XCD more than another, and runs of 4
    // consecutive tiles (neighbouring cells, which share input rows) share an
    // XCD's L2: with x = b % 8, part = (b / 8) % CS and h = b / (8 * CS *
    // NSHARD), the first tile is 32 * (h / 4) + 4 * x + h % 4, a bijection
    // onto [0, G / (NSHARD * CS)) for each part; the parts of a tile share
    // its XCD.
    const int b = (int)blockIdx.x;
    const int part = (b >> 3) % CS;              // cout blocks part*NCBW .. of the tile
    const int shard = ((b >> 3) / CS) % NSHARD;
    const int GS = G / (NSHARD * CS);            // workgroups per segment and part
    const int32_t* seg = plist + (size_t)shard * pcap;
    const int hb = ((b >> 3) / CS) / NSHARD;
    int tile = ((hb >> 2) << 5) + ((b & 7) << 2) + (hb & 3);
    const int n = pcount[shard * CSTRIDE];
    int e = tile * 16 + cl;
    // loads are unconditional, from clamped (always valid) addresses, with the
    // result selected afterwards: a load inside a divergent branch makes the
    // compiler drain every outstanding load at the branch's end
    int qspec = seg[min(e, pcap - 1)];

    if (a.cum_dst && b == 0)
        for (int i = (int)threadIdx.x; i < a.n_cum; i += (int)blockDim.x)
            a.cum_dst[(size_t)i * CSTRIDE] += a.cum_src[(size_t)i * CSTRIDE];

    const bool do_prop = a.has_next && wave == 0 && part == 0;
    while (tile * 16 < n) {
        const bool vrow = e < n;
        const int q = vrow ? qspec : 0;
        const int qimg = q / (a.Hout * a.Wout), ql = q - qimg * (a.Hout * a.Wout);
        const int qr = ql / a.Wout, qc = ql - (ql / a.Wout) * a.Wout;
        const int ibase = qimg * (a.Hin * a.Win);      // first cell of the input image

        // change stamps of the 9 input taps, all in flight together
        uint32_t ev[9];
        int cell[9];
        bool inb[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int ir = S * qr + t / 3 - 1, ic = S * qc + t % 3 - 1;
            inb[t] = vrow && ir >= 0 && ir < a.Hin && ic >= 0 && ic < a.Win;
            cell[t] = ibase + min(max(ir, 0), a.Hin - 1) * a.Win + min(max(ic, 0), a.Win - 1);
            ev[t] = a.stamp_in[cell[t]];
        }
        float* zrow = a.Z + (size_t)q * COUT;
        f4v zo[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
            zo[cb] = *reinterpret_cast<const f4v*>(zrow + min((part * NCBW + cw * NCB + cb) * 16 + 4 * g, COUT - 4));
        // sparse backbones: only a site active now or before can change, and
        // only such sites go to the next layer's list
        bool now = true, prev = true;
        if constexpr (SPARSE) {
            const uint64_t mw = a.memb[q];
            now = memb_now(mw);
            prev = memb_prev(mw, a.epoch);
        }
        PropBatch<4> pb;
        int rows[9];
        bool any[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            rows[t] = (inb[t] && ev[t] == a.epoch) ? cell[t] : -1;
            any[t] = __ballot(rows[t] >= 0) != 0ull;    // no changed input under this tap: skip it
        }
        // sparse, a regular layer followed by another one (SPREAD): the next
        // regular layer's words of the sites whose activity flips, loaded now
        // so that only their swaps end the tile
        MembBatch mbt;
        const bool spread = SPREAD && wave == 0 && part == 0;
        if (spread) memb_issue(a.mnext, q, a.Hout, a.Wout, g == 0 && vrow && now != prev, mbt);

        const char* dbase = static_cast<const char*>(a.delta_in) + g * 16;
        const uint4* wbase = static_cast<const uint4*>(a.wpack) + (size_t)(part * NCBW + cw * NCB) * 64 + lane;
        f4v acc[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = f4v{0.f, 0.f, 0.f, 0.f};

        auto mfma_chunk = [&](const uint4 av, const uint4 (&bv)[NCB]) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                if constexpr (BF16) {
                    bf8v A, B;
                    __builtin_memcpy(&A, &bv[cb], 16);
                    __builtin_memcpy(&B, &av, 16);
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[cb], 0, 0, 0);
                } else {
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].x), __uint_as_float(av.x),
                                                                 acc[cb], 0, 0, 0);
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].y), __uint_as_float(av.y),
                                                                 acc[cb], 0, 0, 0);
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].z), __uint_as_float(av.z),
                                                                 acc[cb], 0, 0, 0);
                    acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv[cb].w), __uint_as_float(av.w),
                                                                 acc[cb], 0, 0, 0);
                }
            }
        };
        static_assert(9 * NCH / KS <= 72, "wider contractions take the wide-layer kernel");
        // narrow inputs: this wavefront's (tap, chunk) steps st = ks + KS*i
        // are fully unrolled and both operands are prefetched PF steps
        // ahead, so the weight and delta loads of later taps overlap the
        // current MFMAs.  The loads are unconditional (clamped step, zero
        // operand past the end): a load under a branch would make the
        // compiler drain every outstanding load where the branch joins.
        constexpr int NSTEP = 9 * NCH;
        constexpr int NSW = (NSTEP + KS - 1) / KS;
        constexpr int PF = NCB == 1 ? 9 : (NCB == 2 ? 8 : 6);
        int srow[NSW];
        bool sany[NSW];
#pragma unroll
        for (int i = 0; i < NSW; ++i) {
            if constexpr (KS == 1) {
                srow[i] = rows[i / NCH];
                sany[i] = any[i / NCH];
            } else {
                const int st = ks + KS * i, t = st / NCH;
                int r = -1;
                bool an = false;
#pragma unroll
                for (int tt = 0; tt < 9; ++tt) {
                    r = t == tt ? rows[tt] : r;
                    an = t == tt ? any[tt] : an;
                }
                srow[i] = st < NSTEP ? r : -1;
                sany[i] = st < NSTEP && an;
            }
        }
        uint4 abuf[NSW];
        uint4 bbuf[NSW][NCB];
        auto issue = [&](int i) {
            const int st = KS == 1 ? i : min(ks + KS * i, NSTEP - 1);
            const int c = st % NCH;
            abuf[i] = *reinterpret_cast<const uint4*>(dbase + (size_t)max(srow[i], 0) * ROWB_IN + c * 64);
            const uint4* wp = wbase + (size_t)((st / NCH) * NCHW + c % NCHW) * NCBT * 64;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) bbuf[i][cb] = wp[cb * 64];
        };
#pragma unroll
        for (int i = 0; i < PF && i < NSW; ++i) issue(i);
        // next layer's change list: the footprint stamps go out after the
        // first steps' operand loads (vector-memory results come back in
        // issue order, so the slower device-scope atomics would otherwise
        // hold up the first matrix instructions); the list positions are
        // taken once step PF's operands, issued after the atomics, have
        // arrived, and the counter's round trip overlaps the remaining steps
        // instead of ending the tile
        if (do_prop) prop_issue<4, false>(a.next, q, vrow && (now || prev), g, a.epoch, pb);
        constexpr int RES = NSW > PF ? PF : NSW - 1;
        PropSlots<4> ps;
#pragma unroll
        for (int i = 0; i < NSW; ++i) {
            if (i + PF < NSW) issue(i + PF);
            uint4 av = abuf[i];
            if (srow[i] < 0) av = make_uint4(0u, 0u, 0u, 0u);
            if constexpr (BF16) {
                const int st = KS == 1 ? i : min(ks + KS * i, NSTEP - 1);
                av = old_half_negated<CIN>(av, st % NCH, g);
            }
            if (sany[i]) mfma_chunk(av, bbuf[i]);
            if (i == RES && do_prop) prop_reserve<4>(a.next, a.epoch, shard, pb, ps);
            // keep the scheduler from hoisting later loads past this step
            __builtin_amdgcn_sched_barrier(0);
        }

        if constexpr (KS > 1) {
            // partial sums of the contraction shares 1..KS-1 into share 0
            __shared__ f4v red[KS - 1][NWC * NCB][64];
            if (ks > 0) {
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) red[ks - 1][cw * NCB + cb][lane] = acc[cb];
            }
            __syncthreads();
            if (ks == 0) {
#pragma unroll
                for (int j = 0; j < KS - 1; ++j)
#pragma unroll
                    for (int cb = 0; cb < NCB; ++cb) {
                        const f4v p = red[j][cw * NCB + cb][lane];
                        acc[cb].x += p.x;
                        acc[cb].y += p.y;
                        acc[cb].z += p.z;
                        acc[cb].w += p.w;
                    }
            }
            __syncthreads();                     // read before the next tile writes
        }
        if (vrow && ks == 0) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int co0 = (part * NCBW + cw * NCB + cb) * 16 + 4 * g;
                if (COUT % 16 == 0 || co0 < COUT) epilogue4<COUT, BF16>(a, q, co0, zo[cb], acc[cb], now, prev);
            }
        }
        if (spread) memb_finish(a.mnext, q, a.Hout, a.Wout, mbt, now ? 1 : -1, a.epoch);
        if (do_prop) prop_write<4>(a.next, shard, pb, ps);

        tile += GS;
        e = tile * 16 + cl;
        if (tile * 16 >= n) break;
        qspec = seg[min(e, pcap - 1)];
    }
}


// ---------------------------------------------------------------------------
// wide layers (more than 4 chunks of 16 input channels per tap)
// ---------------------------------------------------------------------------
// Here one tile's weights (9 * cin * cout values) are far larger than its
// deltas, so a workgroup covers 2 tiles x 2 output-channel blocks (4
// wavefronts, one tile and one block each; the cout dimension is spread over
// NCBT/2 workgroups) and streams both operands tap by tap through LDS with
// asynchronous global->LDS copies: while the matrix cores work on tap t from
// registers, the copies of the next tap are in flight.
// Each copy is shared by the two wavefronts that need it (a vector load of the
// same bytes by every wavefront costs several times more per compute unit).
// Stage layout: [slot][chunk][lane] with slots tile 0, tile 1, block 0,
// block 1; lane l of a 16-byte-per-lane copy lands at base + 16*l, which is
// the MFMA operand layout.  Taps without a changed input in either tile are
// skipped by the whole workgroup.
template <int CIN, int COUT, bool BF16>
struct WideShape {
    static constexpr int KTOT = BF16 ? 2 * CIN : CIN;
    static constexpr int NCH = KTOT / (BF16 ? 32 : 16);    // 1 KB operand chunks per tap
    static constexpr int NCHW = WeightChunks<CIN, BF16>::N; // weight chunks per tap
    static constexpr int NCBT = COUT / 16;
    static constexpr int NH = NCBT / 2;                     // workgroups per tile pair
};

// Groups of four wavefronts over a tile pair's taps: two for a stride-2 layer
// with at most 8 chunks per tap.  Its output list is ~4x shorter than its
// input, so its tile pairs leave compute units idle and a workgroup's tap
// chain ends the launch (c3's 128->256: 192 workgroups).  A stride-1 layer
// has enough tile pairs to fill the chip, and there the larger workgroup
// (one per compute unit at these registers) costs a second round (the
// 504x504 sweep's 128->128: 19.7 -> 24.9 us per launch).
template <int CIN, int COUT, int S, bool BF16>
struct WideGroups {
    static constexpr int KH = S == 2 && WideShape<CIN, COUT, BF16>::NCH <= 8 ? 2 : 1;
};

// plist, pcount, pcap: as for layer_kernel (preloaded copies of a.list,
// a.count, a.cap).
// With KH > 1 the workgroup holds KH groups of the four wavefronts: group k
// contracts the k-th, (k+KH)-th, ... of the tile pair's active taps through
// a stage of its own, so KH taps' copies and matrix work are in flight at
// once, and groups 1..KH-1 add their partial sums into group 0 through LDS,
// in group order.  Every group runs the same number of tap steps (the last
// one idle where the taps do not divide evenly), so the barriers match.
template <int CIN, int COUT, int S, bool BF16, bool SPARSE>
__global__ __launch_bounds__((256 * WideGroups<CIN, COUT, S, BF16>::KH)) void layer_kernel_wide(
    const int32_t* __restrict__ plist, const int32_t* __restrict__ pcount, int pcap, LayerArgs a) {
    using W = WideShape<CIN, COUT, BF16>;
    constexpr int NCH = W::NCH, NCHW = W::NCHW, NCBT = W::NCBT, NH = W::NH, KH = WideGroups<CIN, COUT, S, BF16>::KH;
    constexpr int ROWB_IN = 4 * CIN;
    static_assert(NCH % 2 == 0 && NCHW % 2 == 0 && NCBT % 2 == 0, "shape");
    __shared__ uint4 stage[KH][4][NCH][64];
    __shared__ f4v red[KH > 1 ? KH - 1 : 1][4][64];
    __shared__ int tapmask;

    const int lane = (int)(threadIdx.x & 63u), wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int cl = lane & 15, g = lane >> 4;
    const int kh = wave >> 2, w4 = wave & 3;           // tap group; role in the group
    const int tp = w4 & 1, cbl = w4 >> 1;              // tile and cout block of this wavefront
    const int b = (int)blockIdx.x;
    const int h = b % NH;                              // cout blocks 2h, 2h+1
    const int shard = (b / NH) % NSHARD;
    const int GL = (int)gridDim.x / (NH * NSHARD);     // workgroups per (segment, cout group)
    const int32_t* seg = plist + (size_t)shard * pcap;
    const int n = pcount[shard * CSTRIDE];
    const int cbg = 2 * h + cbl;                       // global cout block of this wavefront
    const bool lead = kh == 0;                         // the group that finishes the tile
    const bool do_prop = a.has_next && h == 0 && cbl == 0 && lead;
    const char* dbase = static_cast<const char*>(a.delta_in) + g * 16;
    const uint4* wbase = static_cast<const uint4*>(a.wpack) + lane;

    for (int pair = (b / NH) / NSHARD; pair * 32 < n; pair += GL) {
        const int e = (2 * pair + tp) * 16 + cl;
        const bool vrow = e < n;
        const int q = vrow ? seg[min(e, pcap - 1)] : 0;
        const int qimg = q / (a.Hout * a.Wout), ql = q - qimg * (a.Hout * a.Wout);
        const int qr = ql / a.Wout, qc = ql - (ql / a.Wout) * a.Wout;
        const int ibase = qimg * (a.Hin * a.Win);
        // the 9 change stamps all in flight together (a ballot between the
        // loads would wait for each in turn)
        uint32_t ev[9];
        int cell[9];
        bool inb[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int ir = S * qr + t / 3 - 1, ic = S * qc + t % 3 - 1;
            inb[t] = vrow && ir >= 0 && ir < a.Hin && ic >= 0 && ic < a.Win;
            cell[t] = ibase + min(max(ir, 0), a.Hin - 1) * a.Win + min(max(ic, 0), a.Win - 1);
            ev[t] = a.stamp_in[cell[t]];
        }
        int rows[9];
        unsigned mask = 0u;
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            rows[t] = (inb[t] && ev[t] == a.epoch) ? cell[t] : -1;
            if (__ballot(rows[t] >= 0) != 0ull) mask |= 1u << t;
        }
        const f4v zo = *reinterpret_cast<const f4v*>(a.Z + (size_t)q * COUT + cbg * 16 + 4 * g);
        bool now = true, prev = true;           // sparse backbones, as in the narrow kernel
        if constexpr (SPARSE) {
            const uint64_t mw = a.memb[q];
            now = memb_now(mw);
            prev = memb_prev(mw, a.epoch);
        }
        PropBatch<4> pb;
        if (do_prop) prop_issue<4, false>(a.next, q, vrow && (now || prev), g, a.epoch, pb);
        if (threadIdx.x == 0) tapmask = 0;
        __syncthreads();
        if (lane == 0 && mask) atomicOr(&tapmask, (int)mask);
        __syncthreads();
        const unsigned taps = (unsigned)__builtin_amdgcn_readfirstlane(tapmask);
        // this group's taps: those with t % KH == kh.  Fixed by the tap index,
        // not by its rank among the tile pair's active taps, so that a cell's
        // partial sums are grouped the same whichever cells share its tile
        // pair (the list order, and with it the pairing, is set by atomics):
        // the maps stay bit-identical from run to run
        unsigned mine = 0u;
        int nsteps = 0;
#pragma unroll
        for (int k = 0; k < KH; ++k) {
            unsigned mk = 0u;
#pragma unroll
            for (int t = k; t < 9; t += KH) mk |= taps & (1u << t);
            if (k == kh) mine = mk;
            nsteps = max(nsteps, __builtin_popcount(mk));
        }

        // copies of tap t into the group's stage: the two wavefronts of a
        // tile share its delta chunks, the two wavefronts of a cout block its
        // weights
        auto issue = [&](int t) __attribute__((always_inline)) {
            const int row = max(rows[t], 0);
#pragma unroll
            for (int c = cbl; c < NCH; c += 2)
                __builtin_amdgcn_global_load_lds(
                    (const __attribute__((address_space(1))) void*)(dbase + (size_t)row * ROWB_IN + c * 64),
                    (__attribute__((address_space(3))) void*)&stage[kh][tp][c][0], 16, 0, 0);
#pragma unroll
            for (int c = tp; c < NCHW; c += 2)
                __builtin_amdgcn_global_load_lds(
                    (const __attribute__((address_space(1))) void*)(wbase + ((size_t)(t * NCHW + c) * NCBT + cbg) * 64),
                    (__attribute__((address_space(3))) void*)&stage[kh][2 + cbl][c][0], 16, 0, 0);
        };

        // one stage buffer per group: a tap's operands move to registers,
        // then the copies of the group's next tap overwrite the stage while
        // the matrix cores work; a small stage lets two workgroups share a
        // compute unit, so one computes while the other waits for its copies
        // take the next layer's list positions now: the counter's round trip
        // then overlaps the taps instead of ending the tile (measured on c3:
        // 364 -> 355 us per stride; the narrow kernel takes them after its
        // first step, since waiting for the footprint atomics before its
        // first loads would delay them)
        PropSlots<4> ps;
        if (do_prop) prop_reserve<4>(a.next, a.epoch, shard, pb, ps);
        f4v acc[1] = {f4v{0.f, 0.f, 0.f, 0.f}};
        if (mine) issue(__builtin_ctz(mine));
        for (int step = 0; step < nsteps; ++step) {
            const bool have = mine != 0u;
            const int t = have ? __builtin_ctz(mine) : 0;
            mine &= mine - 1u;
            __builtin_amdgcn_s_waitcnt(0);             // this wavefront's copies of tap t
            __syncthreads();                           // everyone's copies of tap t
            uint4 av[NCH], bv[NCHW];
            const uint32_t m = have && rows[t] >= 0 ? ~0u : 0u;   // unchanged input: zero row
#pragma unroll
            for (int c = 0; c < NCH; ++c) {
                const uint4 x = stage[kh][tp][c][lane];
                av[c] = make_uint4(x.x & m, x.y & m, x.z & m, x.w & m);
                if constexpr (BF16) av[c] = old_half_negated<CIN>(av[c], c, g);
            }
#pragma unroll
            for (int c = 0; c < NCHW; ++c) bv[c] = stage[kh][2 + cbl][c][lane];
            if (step + 1 < nsteps) {
                __builtin_amdgcn_s_waitcnt(0);         // this wavefront's stage reads are done
                __syncthreads();                       // everyone's: the stages are free
                if (mine) issue(__builtin_ctz(mine));
            }
            if (have) {
#pragma unroll
                for (int c = 0; c < NCH; ++c) {
                    const uint4 bb[1] = {bv[c % NCHW]};
                    mfma_chunk<BF16, 1>(acc, av[c], bb);
                }
            }
        }
        if constexpr (KH > 1) {
            if (!lead) red[kh - 1][w4][lane] = acc[0];
            __syncthreads();
            if (lead) {
#pragma unroll
                for (int k = 0; k < KH - 1; ++k) {
                    const f4v p = red[k][w4][lane];
                    acc[0].x += p.x;
                    acc[0].y += p.y;
                    acc[0].z += p.z;
                    acc[0].w += p.w;
                }
            }
        }
        if (vrow && lead) epilogue4<COUT, BF16>(a, q, cbg * 16 + 4 * g, zo, acc[0], now, prev);
        if constexpr (SPARSE) {
            if (a.mnext.memb && h == 0 && cbl == 0 && g == 0 && lead && vrow && now != prev)
                memb_spread(a.mnext, q, a.Hout, a.Wout, now ? 1 : -1, a.epoch);
        }
        if (do_prop) prop_write<4>(a.next, shard, pb, ps);
        __syncthreads();                               // the stages and partial sums are free again
    }
    if (a.cum_dst && b == 0)
        for (int i = (int)threadIdx.x; i < a.n_cum; i += (int)blockDim.x)
            a.cum_dst[(size_t)i * CSTRIDE] += a.cum_src[(size_t)i * CSTRIDE];
}

// ---------------------------------------------------------------------------
// instantiation table
// ---------------------------------------------------------------------------
#define SSC_CH_LIST(X, CIN, S) X(CIN, 8, S) X(CIN, 16, S) X(CIN, 32, S) X(CIN, 64, S) X(CIN, 128, S) X(CIN, 256, S)
#define SSC_ALL_SHAPES(X)                                                                            \
    SSC_CH_LIST(X, 16, 1) SSC_CH_LIST(X, 32, 1) SSC_CH_LIST(X, 64, 1) SSC_CH_LIST(X, 128, 1)         \
    SSC_CH_LIST(X, 256, 1) SSC_CH_LIST(X, 16, 2) SSC_CH_LIST(X, 32, 2) SSC_CH_LIST(X, 64, 2)         \
    SSC_CH_LIST(X, 128, 2) SSC_CH_LIST(X, 256, 2)

bool layer_supported(int cin, int cout, int stride, bool /*bf16*/) {
#define SSC_SUP(CI, CO, S) if (cin == CI && cout == CO && stride == S) return true;
    SSC_ALL_SHAPES(SSC_SUP)
#undef SSC_SUP
    return false;
}

template <int CI, int CO, int S, bool BF16, bool SPARSE>
static hipError_t launch_shape(const LayerArgs& a, int grid, const LaunchCtx& c) {
    // wide layers: more than 8 input chunks, or more than 4 with at least 8
    // output blocks (a narrow workgroup would then run 2+ blocks x 72 steps
    // per wavefront, on half as many workgroups)
    constexpr int WNCH = WideShape<CI, CO, BF16>::NCH;
    if constexpr ((WNCH > 8 && CO >= 32) || (WNCH > 4 && CO >= 128)) {
        // tile pairs x cout groups x segments; at most ceil(cap / 32) pairs per segment
        constexpr int NH = WideShape<CI, CO, BF16>::NH;
        int gl = std::max(1, grid / (2 * NH * NSHARD));
        gl = std::min(gl, std::max(1, (a.cap + 31) / 32));
        constexpr int KH = WideGroups<CI, CO, S, BF16>::KH;
        return launch_kernel(c, layer_kernel_wide<CI, CO, S, BF16, SPARSE>, dim3(gl * NH * NSHARD), dim3(256 * KH),
                             a.list, a.count, a.cap, a);
    } else {
        // whole runs of 4 tiles on every XCD for every segment and cout part
        using LS = LayerShape<CO, S, BF16 || SPARSE>;
        constexpr int GU = 32 * NSHARD * LS::CS;
        grid = std::max(GU, grid / GU * GU);
        if constexpr (SPARSE)
            if (a.mnext.memb)
                return launch_kernel(c, layer_kernel<CI, CO, S, BF16, true, true>, dim3(grid),
                                     dim3(64 * LS::NW), a.list, a.count, a.cap, a);
        return launch_kernel(c, layer_kernel<CI, CO, S, BF16, SPARSE, false>, dim3(grid), dim3(64 * LS::NW),
                             a.list, a.count, a.cap, a);
    }
}

hipError_t launch_layer(const LayerArgs& a, int cin, int cout, int stride, bool bf16, bool sparse, int grid,
                        const LaunchCtx& c) {
#define SSC_LAUNCH(CI, CO, S)                                                                               \
    if (cin == CI && cout == CO && stride == S) {                                                           \
        if (sparse)                                                                                         \
            return bf16 ? launch_shape<CI, CO, S, true, true>(a, grid, c)                                   \
                        : launch_shape<CI, CO, S, false, true>(a, grid, c);                                 \
        return bf16 ? launch_shape<CI, CO, S, true, false>(a, grid, c)                                      \
                    : launch_shape<CI, CO, S, false, false>(a, grid, c);                                    \
    }
    SSC_ALL_SHAPES(SSC_LAUNCH)
#undef SSC_LAUNCH
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// weight repacking (host)
// ---------------------------------------------------------------------------
size_t wpack_elems(int cin, int cout, bool bf16) {
    return (size_t)9 * (size_t)(bf16 ? std::max(cin, 32) : cin) * (size_t)((cout + 15) / 16 * 16);
}

// Layout, in 16-byte lane vectors: [tap t][chunk c][cout block cb][lane l],
// lane l of block cb holds output channel cb*16 + l%16 and the k-group l/16 of
// chunk c: fp32 k = c*16 + 4*(l/16) + e (e < 4), cin/16 chunks; bf16 k =
// c*32 + 8*(l/16) + e (e < 8), input channel k % cin, max(cin/32, 1) chunks
// (the kernels apply them to both halves of the pair).  Output channels past
// cout (cout = 8) are zero.
void pack_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst) {
    const int ncbt = (cout + 15) / 16;
    if (!bf16) {
        const float* w = static_cast<const float*>(w_oihw);
        float* out = static_cast<float*>(dst);
        const int nch = cin / 16;
        for (int t = 0; t < 9; ++t)
            for (int c = 0; c < nch; ++c)
                for (int cb = 0; cb < ncbt; ++cb)
                    for (int l = 0; l < 64; ++l)
                        for (int e = 0; e < 4; ++e) {
                            const int co = cb * 16 + l % 16;
                            const int ci = c * 16 + 4 * (l / 16) + e;
                            out[((((size_t)t * nch + c) * ncbt + cb) * 64 + l) * 4 + e] =
                                co < cout ? w[(((size_t)co * cin + ci) * 3 + t / 3) * 3 + t % 3] : 0.f;
                        }
    } else {
        const uint16_t* w = static_cast<const uint16_t*>(w_oihw);
        uint16_t* out = static_cast<uint16_t*>(dst);
        const int nch = std::max(cin / 32, 1);
        for (int t = 0; t < 9; ++t)
            for (int c = 0; c < nch; ++c)
                for (int cb = 0; cb < ncbt; ++cb)
                    for (int l = 0; l < 64; ++l)
                        for (int e = 0; e < 8; ++e) {
                            const int co = cb * 16 + l % 16;
                            const int ci = (c * 32 + 8 * (l / 16) + e) % cin;
                            out[((((size_t)t * nch + c) * ncbt + cb) * 64 + l) * 8 + e] =
                                co < cout ? w[(((size_t)co * cin + ci) * 3 + t / 3) * 3 + t % 3] : 0;
                        }
    }
}

}  // namespace ssc
