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
//   * a workgroup owns 16 consecutive cells of A_l and all output channels.
//     For each of the 9 taps it gathers, through the epoch-stamped index map
//     of A_{l-1}, the packed delta rows of the input cells under that tap
//     (rows of unchanged input cells are zero and a tap with no changed input
//     in the whole tile is skipped) and contracts them with the tap's weights
//     on the matrix cores: D[cout x 16 cells] += W_t^T[cout x cin] . dY^T.
//     Summing the 9 taps per output cell in a fixed order is exactly the sum
//     the scatter of Eq. 2 adds into that cell, so the result is
//     deterministic and each Z row is read and written once per stride;
//   * epilogue in registers: Z_new = Z_old + D; store Z_new; emit the next
//     layer's packed delta row (fp32 phi(Z_new) - phi(Z_old), or the bf16 pair
//     [bf16(phi(Z_new)) | bf16(phi(Z_old))]);
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
// Tiles are walked XCD-aware: workgroup b runs on XCD b % 8, and each XCD
// takes a contiguous range of tiles so neighbouring cells (which share input
// rows) meet in the same L2.
#include "device_common.h"

#include <string.h>

namespace ssc {

template <int COUT>
struct LayerShape {
    static constexpr int NCBT = COUT / 16;                  // 16-wide cout blocks
    static constexpr int NW = NCBT >= 4 ? 4 : NCBT;         // wavefronts per workgroup
    static constexpr int NCB = NCBT / NW;                   // cout blocks per wavefront
};

template <int CIN, int COUT, int S, bool BF16>
__global__ __launch_bounds__(64 * LayerShape<COUT>::NW) void layer_kernel(LayerArgs a) {
    constexpr int NCBT = LayerShape<COUT>::NCBT;
    constexpr int NCB = LayerShape<COUT>::NCB;
    constexpr int KTOT = BF16 ? 2 * CIN : CIN;   // contraction length per tap
    constexpr int KCH = BF16 ? 32 : 16;          // k per 64-byte chunk
    constexpr int NCH = KTOT / KCH;
    constexpr int ROWB_IN = 4 * CIN;             // packed input row bytes (fp32, or bf16 pair)
    constexpr int ROWB_OUT = 4 * COUT;

    const int lane = (int)(threadIdx.x & 63u), wave = (int)(threadIdx.x >> 6);
    const int cl = lane & 15, g = lane >> 4;
    const int n = *a.count;

    if (a.cum_dst && blockIdx.x == 0)
        for (int i = (int)threadIdx.x; i < a.n_cum; i += (int)blockDim.x) a.cum_dst[i] += a.cum_src[i];

    const int ntiles = (n + 15) >> 4;
    const int xcd = (int)(blockIdx.x & 7u), slot = (int)(blockIdx.x >> 3);
    const int wgs_per_xcd = (int)(gridDim.x >> 3);
    const int tiles_per_xcd = (ntiles + 7) >> 3;
    for (int k = slot; k < tiles_per_xcd; k += wgs_per_xcd) {
        const int tile = xcd * tiles_per_xcd + k;
        if (tile >= ntiles) break;
        const int e = tile * 16 + cl;
        const bool vrow = e < n;
        const int q = vrow ? a.list[e] : 0;
        const int qr = q / a.Wout, qc = q - (q / a.Wout) * a.Wout;

        f4v acc[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[cb] = f4v{0.f, 0.f, 0.f, 0.f};

        for (int t = 0; t < 9; ++t) {
            const int m = t / 3, nn = t - 3 * (t / 3);
            const int ir = S * qr + m - 1, ic = S * qc + nn - 1;
            int row = -1;
            if (vrow && ir >= 0 && ir < a.Hin && ic >= 0 && ic < a.Win) {
                const uint64_t ev = a.map_in[ir * a.Win + ic];
                if ((uint32_t)(ev >> 32) == a.epoch) row = (int)(uint32_t)ev;
            }
            if (__ballot(row >= 0) == 0ull) continue;   // no changed input under this tap
            const char* arow = static_cast<const char*>(a.delta_in) + (size_t)(row < 0 ? 0 : row) * ROWB_IN + g * 16;
            const uint4* wp = static_cast<const uint4*>(a.wpack) +
                              ((size_t)t * NCH * NCBT + (size_t)wave * NCB) * 64 + lane;
#pragma unroll 2
            for (int c = 0; c < NCH; ++c) {
                uint4 av = make_uint4(0u, 0u, 0u, 0u);
                if (row >= 0) av = *reinterpret_cast<const uint4*>(arow + c * 64);
#pragma unroll
                for (int cb = 0; cb < NCB; ++cb) {
                    const uint4 bv = wp[((size_t)c * NCBT + cb) * 64];
                    if constexpr (BF16) {
                        bf8v A, B;
                        __builtin_memcpy(&A, &bv, 16);
                        __builtin_memcpy(&B, &av, 16);
                        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[cb], 0, 0, 0);
                    } else {
                        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv.x), __uint_as_float(av.x),
                                                                     acc[cb], 0, 0, 0);
                        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv.y), __uint_as_float(av.y),
                                                                     acc[cb], 0, 0, 0);
                        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv.z), __uint_as_float(av.z),
                                                                     acc[cb], 0, 0, 0);
                        acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bv.w), __uint_as_float(av.w),
                                                                     acc[cb], 0, 0, 0);
                    }
                }
            }
        }

        if (vrow) {
            float* zrow = a.Z + (size_t)q * COUT;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int co0 = (wave * NCB + cb) * 16 + 4 * g;
                const f4v zo = *reinterpret_cast<const f4v*>(zrow + co0);
                f4v zn;
                zn.x = zo.x + acc[cb].x;
                zn.y = zo.y + acc[cb].y;
                zn.z = zo.z + acc[cb].z;
                zn.w = zo.w + acc[cb].w;
                *reinterpret_cast<f4v*>(zrow + co0) = zn;
                if (a.delta_out) {
                    f4v yo = zo, yn = zn;
                    if (a.relu) {
                        yo.x = fmaxf(yo.x, 0.f); yo.y = fmaxf(yo.y, 0.f); yo.z = fmaxf(yo.z, 0.f); yo.w = fmaxf(yo.w, 0.f);
                        yn.x = fmaxf(yn.x, 0.f); yn.y = fmaxf(yn.y, 0.f); yn.z = fmaxf(yn.z, 0.f); yn.w = fmaxf(yn.w, 0.f);
                    }
                    char* drow = static_cast<char*>(a.delta_out) + (size_t)e * ROWB_OUT;
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
            }
        }
        if (a.has_next && wave == 0) propagate_cells<4>(a.next, vrow ? q : -1, g, a.epoch);
    }
}

// ---------------------------------------------------------------------------
// instantiation table
// ---------------------------------------------------------------------------
#define SSC_CH_LIST(X, CIN, S) X(CIN, 16, S) X(CIN, 32, S) X(CIN, 64, S) X(CIN, 128, S) X(CIN, 256, S)
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

hipError_t launch_layer(const LayerArgs& a, int cin, int cout, int stride, bool bf16, int grid, hipStream_t s) {
    grid = grid < 8 ? 8 : (grid & ~7);
#define SSC_LAUNCH(CI, CO, S)                                                                               \
    if (cin == CI && cout == CO && stride == S) {                                                           \
        dim3 blk(64 * LayerShape<CO>::NW);                                                                  \
        if (bf16) hipLaunchKernelGGL((layer_kernel<CI, CO, S, true>), dim3(grid), blk, 0, s, a);             \
        else hipLaunchKernelGGL((layer_kernel<CI, CO, S, false>), dim3(grid), blk, 0, s, a);                 \
        return hipGetLastError();                                                                           \
    }
    SSC_ALL_SHAPES(SSC_LAUNCH)
#undef SSC_LAUNCH
    return hipErrorInvalidValue;
}

// ---------------------------------------------------------------------------
// weight repacking (host)
// ---------------------------------------------------------------------------
size_t wpack_elems(int cin, int cout, bool bf16) {
    return (size_t)9 * (size_t)(bf16 ? 2 * cin : cin) * (size_t)cout;
}

// Layout, in 16-byte lane vectors: [tap t][chunk c][cout block cb][lane l],
// lane l of block cb holds output channel cb*16 + l%16 and the k-group l/16 of
// chunk c: fp32 k = c*16 + 4*(l/16) + e (e < 4); bf16 k = c*32 + 8*(l/16) + e
// (e < 8) over the pair [W | -W].
void pack_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst) {
    const int ncbt = cout / 16;
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
                                w[(((size_t)co * cin + ci) * 3 + t / 3) * 3 + t % 3];
                        }
    } else {
        const uint16_t* w = static_cast<const uint16_t*>(w_oihw);
        uint16_t* out = static_cast<uint16_t*>(dst);
        const int nch = (2 * cin) / 32;
        for (int t = 0; t < 9; ++t)
            for (int c = 0; c < nch; ++c)
                for (int cb = 0; cb < ncbt; ++cb)
                    for (int l = 0; l < 64; ++l)
                        for (int e = 0; e < 8; ++e) {
                            const int co = cb * 16 + l % 16;
                            const int k = c * 32 + 8 * (l / 16) + e;
                            const int ci = k < cin ? k : k - cin;
                            uint16_t v = w[(((size_t)co * cin + ci) * 3 + t / 3) * 3 + t % 3];
                            if (k >= cin) v ^= 0x8000u;   // -W: exact sign flip
                            out[((((size_t)t * nch + c) * ncbt + cb) * 64 + l) * 8 + e] = v;
                        }
    }
}

}  // namespace ssc
