// Wide stride-1 layers in two launches.
//
// Method (SSCATeR, arXiv 2512.08557, Eq. 2): a changed input site p scatters
// (I_curr - I_prev)[p] x W[m, n] into the output site (i - m + 1, j - n + 1)
// for each of the nine taps.  For the 128- and 256-channel layers of the
// backbone this is done as the scatter form of the contraction, a dense
// product over the changed rows only:
//
//   contract_kernel   part[p][tap][co] = sum_ci dY[p][ci] * W[co][ci][tap]
//                     for every p in A_{l-1}: [|A_{l-1}| x cin] x [cin x 9*cout]
//                     on the matrix cores;
//   tap_sum_kernel    for every q in A_l: Z[q] += sum over the taps whose input
//                     p(q, tap) changed of part[p][tap], in the fixed order
//                     tap = 0..8; then the delta epilogue of the next layer and
//                     the propagation of A_l to the next layer's list.
//
// The product's rows are the changed cells, so it carries exactly the
// method's work (no zero rows, unlike an output-stationary tile whose cells
// changed under different taps), and every row of it is a dense 64-row x
// 64-column tile of a plain GEMM.  The sum is output-stationary with plain
// stores: deterministic, and each Z row is read and written once.  The
// contributions travel through HBM once (written by the product, read by the
// sum), which is the gather-GEMM-scatter structure of the paper's own kernel
// (Sec. V) with the scatter made a gather, so no atomics touch the maps.
//
// contract_kernel, per workgroup tile (64 changed rows x 64 columns, 4
// wavefronts of 32 x 32): the input channels stream in 128-byte chunks
// through a ring of LDS stages filled by asynchronous global->LDS copies, the
// copies of the next chunks in flight while the matrix cores work on the
// current one.  Operand layout in a stage: [row][8 x 16 bytes], the 16-byte
// piece c of row r stored in slot c ^ ((r >> 1) & 7), so that the rows a
// wavefront reads at one k are spread over all 64 LDS banks.
//   fp32: v_mfma_f32_32x32x2_f32, lane l supplies row l%32 at k = 4*(l/32)+e
//         of an 8-k group (e = 0..3 over four instructions);
//   bf16: the delta is the exact pair [Y_new | Y_old] (bf16 values), and
//         v_mfma_f32_32x32x16_bf16 contracts both halves with the same weight
//         chunk into two fp32 accumulators, differenced at the end: the
//         weights move once, not as a [W | -W] pair.
//   D: lane l holds column l%32 and rows 8*(r/4) + 4*(l/32) + r%4, r = 0..15.
#include "device_common.h"

#include <algorithm>
#include <cstring>

namespace ssc {

typedef float f16v __attribute__((ext_vector_type(16)));

template <int CIN, int COUT, bool BF16>
struct CShape {
    static constexpr int ESZ = BF16 ? 2 : 4;         // bytes of a stored element
    static constexpr int N = 9 * COUT;               // product columns: (tap, output channel)
    static constexpr int NT = N / 64;                // 64-column tiles
    // rows per tile: 64 (four wavefronts of 32 x 32).  Measured against
    // 32-row tiles (two wavefronts, six workgroups per compute unit): the
    // same launch time, at twice the weight traffic from L2
    static constexpr int MT = 64;
    static constexpr int NW = 2 * MT / 32;           // wavefronts: MT/32 x 2 quadrants of 32 x 32
    static constexpr int NCH = CIN * ESZ / 128;      // 128-byte chunks of a cin row
    static constexpr int NA = BF16 ? 2 : 1;          // A operands: the fp32 delta, or the new and old halves
    static constexpr int ROWB = 4 * CIN;             // bytes of an input delta row
    static constexpr int WROWB = CIN * ESZ;          // bytes of a weight row
    static constexpr int OPA = MT * 128;             // one A operand of one chunk: MT rows x 128 bytes
    static constexpr int OPBB = 64 * 128;            // the B operand of one chunk: 64 rows x 128 bytes
    static constexpr int STB = NA * OPA + OPBB;      // one stage
    // stages in the ring: 48 KB of LDS, so three workgroups share a compute
    // unit and the ~400-650 tiles of a 432x496 backbone layer are resident at
    // once (with 64 KB, two per unit, a second round of tiles started only as
    // the first ended); fp32 keeps two chunks in flight behind the one being
    // contracted, bf16 (24 KB per stage) one
    static constexpr int S = BF16 ? 2 : 3;
    static constexpr int BPW = 8 / NW;               // B blocks (1 KB) each wavefront copies per chunk
    static constexpr int LPC = 2 * NA + BPW;         // copies per thread per chunk
    static constexpr int SLOTS = 768;                // resident workgroups on 256 compute units
    // slot of the 16-byte piece c of row r: c ^ ((r >> 1) & 7).  gfx950's LDS
    // has 64 banks (256 bytes), so the 16 lanes served together (rows i ..
    // i+15 of one piece) must fall in 16 different 16-byte bank groups: row
    // r lands in the half r & 1 of the 256 bytes, and the xor with (r >> 1) & 7
    // spreads rows of equal parity over the 8 groups of that half.  (The xor
    // with r & 7 leaves rows 8 apart in the same group: measured
    // SQ_LDS_BANK_CONFLICT / active cycles 0.89 against 0 now, at the same
    // launch time, the loop being bound by the matrix cores.)
    static constexpr int SWZ = 1;
    static_assert(N % 64 == 0 && NCH >= 2, "shape");
};

// plist, pcount, pcap: preloaded copies of a.list, a.count, a.cap.
template <int CIN, int COUT, bool BF16>
__global__ __launch_bounds__((64 * CShape<CIN, COUT, BF16>::NW)) void contract_kernel(
    const int32_t* __restrict__ plist, const int32_t* __restrict__ pcount, int pcap, ContractArgs a) {
    using C = CShape<CIN, COUT, BF16>;
    constexpr int MT = C::MT, NW = C::NW;
    // one LDS array per stage: the compiler then tracks the copies into each
    // stage separately and waits only for those a read depends on
    __shared__ __attribute__((aligned(1024))) char st0[C::STB];
    __shared__ __attribute__((aligned(1024))) char st1[C::S > 1 ? C::STB : 16];
    __shared__ __attribute__((aligned(1024))) char st2[C::S > 2 ? C::STB : 16];
    __shared__ int rowcell[MT];

    const int tid = (int)threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w % (MT / 32), wn = w / (MT / 32);  // this wavefront's 32 x 32 quadrant
    const int li = lane & 31, kg = lane >> 5;
    const int n0 = pcount[0], n1 = pcount[CSTRIDE];
    const int mt0 = (n0 + MT - 1) / MT;
    const int total = (mt0 + (n1 + MT - 1) / MT) * C::NT;
    // copy roles: 1 KB blocks of 8 rows; wavefront w fills A blocks w and
    // NW + w, and B blocks w + j*NW; lane l takes row 8k + l/8 of block k and
    // the 16-byte piece of it that belongs in slot l % 8
    const int cr = lane >> 3;
    // the piece lane l copies into slot l % 8 of row 8k + l/8
    auto piece = [&](int k) { return ((lane & 7) ^ (((8 * k + cr) >> C::SWZ) & 7)) * 16; };
    const char* dsrc = static_cast<const char*>(a.delta_in);
    const char* wsrc = static_cast<const char*>(a.wg);

    for (int t = (int)blockIdx.x; t < total; t += (int)gridDim.x) {
        // tile t: 64-column block t % NT of M-tile t / NT, the M-tiles of
        // list segment 0 first (an order with the segments interleaved, so
        // that a tile's list entries can be loaded before the counts are
        // known, measured 0.5-1 us slower per launch)
        const int mt = t / C::NT, nt = t - mt * C::NT;
        const int seg = mt < mt0 ? 0 : 1;
        const int base = (mt - (seg ? mt0 : 0)) * MT;
        const int nseg = seg ? n1 : n0;
        const int32_t* lst = plist + (size_t)seg * pcap;
        // rows past the segment's end copy row `base` (always valid) and are
        // never stored: a row of the product depends on its own A row only
        const int r0 = 8 * w + cr, r1 = 8 * (NW + w) + cr;
        const int cell0 = lst[base + (base + r0 < nseg ? r0 : 0)];
        const int cell1 = lst[base + (base + r1 < nseg ? r1 : 0)];
        if (tid < MT) rowcell[tid] = base + tid < nseg ? lst[base + tid] : -1;
        const char* a0 = dsrc + (size_t)cell0 * C::ROWB + piece(w);
        const char* a1 = dsrc + (size_t)cell1 * C::ROWB + piece(NW + w);
        const char* bsrc = wsrc + (size_t)(nt * 64 + cr) * C::WROWB;

        auto issue = [&](int c, char* stp) __attribute__((always_inline)) {
            char* d0 = stp + w * 1024;
            char* d1 = stp + (NW + w) * 1024;
            copy16(a0 + c * 128, d0);
            copy16(a1 + c * 128, d1);
            if constexpr (BF16) {   // the old half of the pair row
                copy16(a0 + 2 * CIN + c * 128, d0 + C::OPA);
                copy16(a1 + 2 * CIN + c * 128, d1 + C::OPA);
            }
#pragma unroll
            for (int j = 0; j < C::BPW; ++j) {
                const int k = w + j * NW;            // B block: rows 8k .. 8k+7
                copy16(bsrc + (size_t)(8 * k) * C::WROWB + piece(k) + c * 128, stp + C::NA * C::OPA + k * 1024);
            }
        };
        auto stage = [&](int k) -> char* { return k == 0 ? st0 : (k == 1 ? st1 : st2); };

        f16v acc = {};
        f16v acc_old = {};
        const int ra = 32 * wm + li, rb = 32 * wn + li;
        auto compute = [&](const char* stp) __attribute__((always_inline)) {
            // the chunk's operands first (all LDS reads in flight together),
            // then its matrix instructions
            uint4 av[4], bv[4], ov[4];
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c16 = 2 * g + kg;
                const int sa = 16 * (c16 ^ ((ra >> C::SWZ) & 7)), sb = 16 * (c16 ^ ((rb >> C::SWZ) & 7));
                av[g] = *reinterpret_cast<const uint4*>(stp + ra * 128 + sa);
                bv[g] = *reinterpret_cast<const uint4*>(stp + C::NA * C::OPA + rb * 128 + sb);
                if constexpr (BF16) ov[g] = *reinterpret_cast<const uint4*>(stp + C::OPA + ra * 128 + sa);
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                if constexpr (BF16) {
                    bf8v A, O, B;
                    __builtin_memcpy(&A, &av[g], 16);
                    __builtin_memcpy(&O, &ov[g], 16);
                    __builtin_memcpy(&B, &bv[g], 16);
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A, B, acc, 0, 0, 0);
                    acc_old = __builtin_amdgcn_mfma_f32_32x32x16_bf16(O, B, acc_old, 0, 0, 0);
                } else {
                    const uint4 x = av[g], y = bv[g];
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.x), __uint_as_float(y.x), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.y), __uint_as_float(y.y), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.z), __uint_as_float(y.z), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(x.w), __uint_as_float(y.w), acc, 0, 0, 0);
                }
            }
        };

        // the ring: chunks 0 .. S-2 in flight before the first wait
#pragma unroll
        for (int c = 0; c < C::S - 1; ++c) issue(c, stage(c));
#pragma unroll
        for (int c = 0; c < C::NCH; ++c) {
            // this thread's copies of chunk c have landed (the copies of the
            // later chunks already issued may still be in flight) ...
            const int ahead = min(C::S - 2, C::NCH - 1 - c);
            wait_vm_n(max(ahead, 0) * C::LPC);
            // ... and everyone's; everyone is also done reading chunk c - 1,
            // whose stage the next copies overwrite
            lds_barrier();
            if (c + C::S - 1 < C::NCH) issue(c + C::S - 1, stage((c + C::S - 1) % C::S));
            asm volatile("" ::: "memory");   // the copies go out before the chunk's reads
            compute(stage(c % C::S));
        }

        // D: column n = nt*64 + 32*wn + li, rows 32*wm + 8*(r/4) + 4*kg + r%4
        float* out = a.part + (size_t)(nt * 64 + 32 * wn + li);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * wm + 8 * (r >> 2) + 4 * kg + (r & 3);
            const int cell = rowcell[row];
            const float v = BF16 ? acc[r] - acc_old[r] : acc[r];
            // non-temporal: the contributions are read once, by the tap sum,
            // so they are not kept in L2 (which the end of the launch would
            // otherwise have to write back); measured c3 289 -> 271 us per
            // stride together with the non-temporal loads of the tap sum
            if (cell >= 0) __builtin_nontemporal_store(v, out + (size_t)cell * C::N);
        }
        lds_barrier();     // the stages and the row table are free for the next tile
    }
}

// Output-stationary sum of the tap contributions.  A workgroup owns
// TC = 4 * CPI consecutive cells of one list segment, wavefront w the CPI
// cells w*CPI .. : COUT/4 lanes per cell, 4 channels per lane, each tap's row
// a coalesced 16-byte load per lane (the zero row for a tap whose input did
// not change), all of a cell's loads in flight together.  Propagation: 16
// lanes per cell, one tap slot each, wavefront w for cells 4w .. 4w+3.
template <int COUT>
struct TapShape {
    static constexpr int LPC = COUT / 4;         // lanes per cell
    static constexpr int CPI = 64 / LPC;         // cells per wavefront
    static constexpr int TC = 4 * CPI;           // cells per workgroup tile
};

template <int COUT, bool BF16, bool SPARSE>
__global__ __launch_bounds__(256) void tap_sum_kernel(const int32_t* __restrict__ plist,
                                                       const int32_t* __restrict__ pcount, int pcap, LayerArgs a) {
    constexpr int N = 9 * COUT;
    constexpr int LPC = TapShape<COUT>::LPC, CPI = TapShape<COUT>::CPI, TC = TapShape<COUT>::TC;
    static_assert(COUT % 64 == 0 && COUT <= 256, "tap sum shape");

    const int lane = (int)(threadIdx.x & 63u);
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int b = (int)blockIdx.x, G = (int)gridDim.x;   // G a multiple of 16
    // segment (b / 8) % 2; within a segment the workgroups of all eight XCDs
    // take consecutive tiles
    const int shard = (b >> 3) & 1;
    const int GS = G >> 1;
    int tile = ((b >> 4) << 3) | (b & 7);
    const int32_t* seg = plist + (size_t)shard * pcap;
    const int n = pcount[shard * CSTRIDE];

    if (a.cum_dst && b == 0)
        for (int i = (int)threadIdx.x; i < a.n_cum; i += (int)blockDim.x)
            a.cum_dst[(size_t)i * CSTRIDE] += a.cum_src[(size_t)i * CSTRIDE];

    const int sub = lane & 15;                   // propagation: tap slot of the lane
    const int cp = 4 * w + (lane >> 4);          // propagation: cell of the lane (cp < TC)
    const bool prop_wave = 4 * w < TC;
    const int co0 = 4 * (lane % LPC);            // channel work: first channel of the lane
    const int cc = w * CPI + lane / LPC;         // channel work: cell of the lane
    for (;; tile += GS) {
        const int t0 = tile * TC;
        // the cell of the channel work, the propagation cell and the tile's
        // first cell, from clamped (always valid) positions, loaded together
        // with the count on the first pass
        const int e = t0 + cc, ep = t0 + cp;
        const int qs = seg[min(e, pcap - 1)], qps = seg[min(ep, pcap - 1)], q0 = seg[min(t0, pcap - 1)];
        if (t0 >= n) break;
        const bool vrow = e < n;
        const int q = vrow ? qs : q0;
        const bool vp = prop_wave && ep < n;
        const int qp = vp ? qps : q0;
        const f4v zo = *reinterpret_cast<const f4v*>(a.Z + (size_t)q * COUT + co0);
        bool now = true, prev = true, nowp = true, prevp = true;
        if constexpr (SPARSE) {
            const uint64_t mw = a.memb[q], mwp = a.memb[qp];
            now = memb_now(mw);
            prev = memb_prev(mw, a.epoch);
            nowp = memb_now(mwp);
            prevp = memb_prev(mwp, a.epoch);
        }
        const int qimg = q / (a.Hout * a.Wout), ql = q - qimg * (a.Hout * a.Wout);
        const int qr = ql / a.Wout, qc = ql - (ql / a.Wout) * a.Wout;
        const int ibase = qimg * (a.Hin * a.Win);
        // tap t = 3m + n: input (qr + m - 1, qc + n - 1), its row t of part
        uint32_t ev[9];
        int cell[9];
        bool inb[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int ir = qr + t / 3 - 1, ic = qc + t % 3 - 1;
            inb[t] = ir >= 0 && ir < a.Hin && ic >= 0 && ic < a.Win;
            cell[t] = ibase + min(max(ir, 0), a.Hin - 1) * a.Win + min(max(ic, 0), a.Win - 1);
            ev[t] = a.stamp_in[cell[t]];
        }
        // the next layer's footprint stamps go out in the same round trip
        PropBatch<16> pb;
        if (a.has_next && prop_wave) prop_issue<16, false>(a.next, qp, vp && (nowp || prevp), sub, a.epoch, pb);
        f4v v[9];
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const bool ch = inb[t] && ev[t] == a.epoch;
            const float* src = (ch ? a.part + (size_t)cell[t] * N : a.zero) + t * COUT + co0;
            v[t] = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(src));
        }
        // take the next layer's list positions now: the counter's round trip
        // then overlaps the contributions' instead of ending the tile
        PropSlots<16> ps;
        if (a.has_next && prop_wave) prop_reserve<16>(a.next, a.epoch, shard, pb, ps);
        f4v d = v[0];
#pragma unroll
        for (int t = 1; t < 9; ++t) {
            d.x += v[t].x;
            d.y += v[t].y;
            d.z += v[t].z;
            d.w += v[t].w;
        }
        if (vrow) epilogue4<COUT, BF16>(a, q, co0, zo, d, now, prev);
        if constexpr (SPARSE) {
            if (a.mnext.memb && sub == 0 && vp && nowp != prevp)
                memb_spread(a.mnext, qp, a.Hout, a.Wout, nowp ? 1 : -1, a.epoch);
        }
        if (a.has_next && prop_wave) prop_write<16>(a.next, shard, pb, ps);
    }
}

// ---------------------------------------------------------------------------
// shapes and launchers
// ---------------------------------------------------------------------------
#define SSC_CONTRACT_SHAPES(X) X(128, 128) X(128, 256) X(256, 128) X(256, 256)

bool contract_supported(int cin, int cout, int stride, bool /*bf16*/) {
    if (stride != 1) return false;
#define SSC_CSUP(CI, CO) if (cin == CI && cout == CO) return true;
    SSC_CONTRACT_SHAPES(SSC_CSUP)
#undef SSC_CSUP
    return false;
}

template <int CI, int CO, bool BF16>
static hipError_t launch_ct(const ContractArgs& a, int grid, const LaunchCtx& c) {
    using C = CShape<CI, CO, BF16>;
    // as many workgroups as are resident at once; a larger list loops over
    // its remaining tiles
    (void)grid;
    grid = C::SLOTS;
    return launch_kernel(c, contract_kernel<CI, CO, BF16>, dim3(grid), dim3(64 * C::NW), a.list, a.count, a.cap, a);
}

hipError_t launch_contract(const ContractArgs& a, int cin, int cout, bool bf16, int grid, const LaunchCtx& c) {
#define SSC_CL(CI, CO) \
    if (cin == CI && cout == CO) return bf16 ? launch_ct<CI, CO, true>(a, grid, c) : launch_ct<CI, CO, false>(a, grid, c);
    SSC_CONTRACT_SHAPES(SSC_CL)
#undef SSC_CL
    return hipErrorInvalidValue;
}

template <int CO, bool BF16, bool SPARSE>
static hipError_t launch_ts(const LayerArgs& a, int grid, const LaunchCtx& c) {
    return launch_kernel(c, tap_sum_kernel<CO, BF16, SPARSE>, dim3(grid), dim3(256), a.list, a.count, a.cap, a);
}

hipError_t launch_tap_sum(const LayerArgs& a, int cout, bool bf16, bool sparse, int grid, const LaunchCtx& c) {
    grid = std::max(16, grid / 16 * 16);
#define SSC_TS(CO)                                                                            \
    if (cout == CO) {                                                                         \
        if (sparse) return bf16 ? launch_ts<CO, true, true>(a, grid, c) : launch_ts<CO, false, true>(a, grid, c); \
        return bf16 ? launch_ts<CO, true, false>(a, grid, c) : launch_ts<CO, false, false>(a, grid, c);           \
    }
    SSC_TS(128)
    SSC_TS(256)
#undef SSC_TS
    return hipErrorInvalidValue;
}

// [9*cout][cin]: row n = tap*cout + co holds W[co][ci][tap/3][tap%3] over ci.
void pack_contract_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst) {
    for (int t = 0; t < 9; ++t)
        for (int co = 0; co < cout; ++co)
            for (int ci = 0; ci < cin; ++ci) {
                const size_t from = (((size_t)co * cin + ci) * 3 + t / 3) * 3 + t % 3;
                const size_t to = ((size_t)t * cout + co) * cin + ci;
                if (bf16)
                    static_cast<uint16_t*>(dst)[to] = static_cast<const uint16_t*>(w_oihw)[from];
                else
                    static_cast<float*>(dst)[to] = static_cast<const float*>(w_oihw)[from];
            }
}

}  // namespace ssc
