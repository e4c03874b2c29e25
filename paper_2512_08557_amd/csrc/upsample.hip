// Upsampling neck: transposed convolution with kernel = stride S on a backbone
// block's output, on the changed cells only, into the persistent concatenated
// neck map (Sec. III-B, backbone paragraph: the blocks are upsampled and
// concatenated; Alg. 1, deconvolution branch: every upsampled site under a
// changed site is changed).
//
// Kernel = stride, so output cell (S*i + a, S*j + b) has exactly one input
// cell (i, j):  Z[S*i + a][S*j + b][co] += sum_ci dY[i][j][ci] * W[ci][co][a][b].
// The delta form of Eq. 2 for this operator touches only the S x S block of
// each changed input cell, each output cell is written by one workgroup, and
// no atomics are needed.  The work list is the source layer's change list.
//
// Per changed input cell the contraction is [cin] x [cin x S*S*cout]: output
// block ob = (a*S + b)*NCBT + cb holds 16 output channels of one sub-cell.
// A workgroup takes tiles of 16 input cells for 4*BPW output blocks (4
// wavefronts, BPW blocks each).  A tile's delta rows (the B operand of every
// block) are copied once into LDS with asynchronous global->LDS copies shared
// by the four wavefronts; each wavefront loads the weights of its blocks once
// and keeps them in registers for all its tiles (they do not depend on the
// tile), and the launch holds about two workgroups per compute unit, so that
// each takes several tiles of a long list.
#include "device_common.h"

#include <algorithm>

namespace ssc {

template <int CIN, int COUT, int S, bool BF16>
struct UpShape {
    static constexpr int KTOT = BF16 ? 2 * CIN : CIN;
    static constexpr int NCH = KTOT / (BF16 ? 32 : 16);   // 1 KB operand chunks
    static constexpr int NCBT = COUT / 16;
    static constexpr int NOB = S * S * NCBT;              // output blocks per input cell
    static constexpr int BPW = NOB >= 8 ? 2 : 1;          // output blocks per wavefront
    static constexpr int OBG = (NOB + 4 * BPW - 1) / (4 * BPW);   // workgroups per tile
};

template <int CIN, int COUT, int S, bool BF16>
__global__ __launch_bounds__(256) void upsample_kernel(UpArgs a) {
    using U = UpShape<CIN, COUT, S, BF16>;
    constexpr int NCH = U::NCH, NOB = U::NOB, NCBT = U::NCBT, BPW = U::BPW, OBG = U::OBG;
    constexpr int ROWB = 4 * CIN;                          // delta row bytes (fp32, or bf16 pair)
    __shared__ uint4 As0[NCH][64];
    __shared__ uint4 As1[NCH][64];

    const int lane = (int)(threadIdx.x & 63u), wave = (int)(threadIdx.x >> 6);
    const int cl = lane & 15, g = lane >> 4;
    const int b = (int)blockIdx.x;
    const int og = b % OBG;
    const int shard = (b / OBG) % NSHARD;
    const int TG = (int)gridDim.x / (OBG * NSHARD);        // workgroups per (segment, block group)
    const int32_t* seg = a.list + (size_t)shard * a.cap;
    const int n = a.count[shard * CSTRIDE];
    const char* dbase = static_cast<const char*>(a.delta_src) + g * 16;
    const uint4* wbase = static_cast<const uint4*>(a.wpack) + lane;
    const int Wn = S * a.Wsrc;

    int ob[BPW];
    bool obv[BPW];
#pragma unroll
    for (int k = 0; k < BPW; ++k) {
        const int o = (og * 4 + wave) * BPW + k;
        obv[k] = o < NOB;
        ob[k] = obv[k] ? o : 0;
    }
    // this wavefront's weights, for every tile
    uint4 bw[BPW][NCH];
    if ((b / OBG) / NSHARD * 16 < n) {
#pragma unroll
        for (int k = 0; k < BPW; ++k)
#pragma unroll
            for (int c = 0; c < NCH; ++c) bw[k][c] = wbase[((size_t)c * NOB + ob[k]) * 64];
    }

    // tiles tile0, tile0 + TG, ...: the next tile's delta rows (into the other
    // LDS buffer) and old Z values go out before this tile's matrix work, and
    // the list entry of the tile after it too, so that only the first tile
    // waits for its loads.  The two buffers are separate arrays and the loop
    // takes two tiles per pass, so that the compiler sees a tile's reads and
    // the next tile's copies touch different arrays (with one array indexed
    // at run time it waits for every copy before the reads)
    auto entry = [&](int t) {
        const int e = t * 16 + cl;
        return e < n ? seg[min(e, a.cap - 1)] : 0;
    };
    auto out_cell = [&](int p, int k) {
        const int i = p / a.Wsrc, j = p - (p / a.Wsrc) * a.Wsrc;
        const int ab = ob[k] / NCBT;
        return (S * i + ab / S) * Wn + (S * j + ab % S);
    };
    auto z_at = [&](int oc, int k) {
        const int cb = ob[k] - (ob[k] / NCBT) * NCBT;
        return a.Z + (size_t)oc * a.ctot + a.coff + cb * 16 + 4 * g;
    };
    int tile = (b / OBG) / NSHARD;
    int pc = 0, pn = 0;        // cells of this lane's row in this tile and the next
    f4v zo[BPW];
    if (tile * 16 < n) {
        pc = entry(tile);
#pragma unroll
        for (int c = wave; c < NCH; c += 4)
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(dbase + (size_t)pc * ROWB + c * 64),
                (__attribute__((address_space(3))) void*)&As0[c][0], 16, 0, 0);
#pragma unroll
        for (int k = 0; k < BPW; ++k) zo[k] = *reinterpret_cast<const f4v*>(z_at(out_cell(pc, k), k));
        pn = entry(tile + TG);
    }
    // one tile from `cur`, the next one's rows into `nxt`; false past the end
    auto step = [&](uint4 (&cur)[NCH][64], uint4 (&nxt)[NCH][64]) __attribute__((always_inline)) {
        if (tile * 16 >= n) return false;
        const bool vrow = tile * 16 + cl < n;
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();                                   // this tile's chunks have landed; `nxt` is free
        const bool more = (tile + TG) * 16 < n;
        f4v zn_next[BPW];
        int pnn = 0;
        if (more) {
#pragma unroll
            for (int c = wave; c < NCH; c += 4)
                __builtin_amdgcn_global_load_lds(
                    (const __attribute__((address_space(1))) void*)(dbase + (size_t)pn * ROWB + c * 64),
                    (__attribute__((address_space(3))) void*)&nxt[c][0], 16, 0, 0);
#pragma unroll
            for (int k = 0; k < BPW; ++k) zn_next[k] = *reinterpret_cast<const f4v*>(z_at(out_cell(pn, k), k));
            pnn = entry(tile + 2 * TG);
        }
        f4v acc[BPW];
#pragma unroll
        for (int k = 0; k < BPW; ++k) acc[k] = f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const uint4 av = cur[c][lane];
#pragma unroll
            for (int k = 0; k < BPW; ++k) {
                if constexpr (BF16) {
                    bf8v A, B;
                    __builtin_memcpy(&A, &bw[k][c], 16);
                    __builtin_memcpy(&B, &av, 16);
                    acc[k] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, B, acc[k], 0, 0, 0);
                } else {
                    acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw[k][c].x), __uint_as_float(av.x), acc[k], 0, 0, 0);
                    acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw[k][c].y), __uint_as_float(av.y), acc[k], 0, 0, 0);
                    acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw[k][c].z), __uint_as_float(av.z), acc[k], 0, 0, 0);
                    acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(bw[k][c].w), __uint_as_float(av.w), acc[k], 0, 0, 0);
                }
            }
        }
        if (vrow) {
#pragma unroll
            for (int k = 0; k < BPW; ++k) {
                if (!obv[k]) continue;
                f4v zn;
                zn.x = zo[k].x + acc[k].x;
                zn.y = zo[k].y + acc[k].y;
                zn.z = zo[k].z + acc[k].z;
                zn.w = zo[k].w + acc[k].w;
                const int oc = out_cell(pc, k);
                *reinterpret_cast<f4v*>(z_at(oc, k)) = zn;
                if (g == 0) a.stamp[oc] = a.epoch;         // every writer stores the same value
            }
        }
        if (more) {
#pragma unroll
            for (int k = 0; k < BPW; ++k) zo[k] = zn_next[k];
        }
        pc = pn;
        pn = pnn;
        tile += TG;
        return true;
    };
    while (step(As0, As1) && step(As1, As0)) {
    }
}

#define SSC_UP_SHAPES(X)                                                                                    \
    X(64, 128, 1) X(64, 64, 1) X(64, 32, 1) X(64, 16, 1) X(128, 128, 2) X(128, 64, 2) X(128, 128, 1)        \
    X(256, 128, 4) X(256, 64, 4) X(256, 128, 2) X(32, 32, 1) X(32, 32, 2) X(16, 16, 1) X(16, 16, 2)          \
    X(16, 32, 2) X(16, 16, 4) X(32, 16, 4) X(64, 32, 2) X(64, 64, 2) X(64, 64, 4)

bool upsample_supported(int cin, int cout, int stride) {
#define SSC_SUP(CI, CO, S) if (cin == CI && cout == CO && stride == S) return true;
    SSC_UP_SHAPES(SSC_SUP)
#undef SSC_SUP
    return false;
}

template <int CI, int CO, int S, bool BF16>
static hipError_t launch_up_shape(const UpArgs& a, int grid, const LaunchCtx& c) {
    using U = UpShape<CI, CO, S, BF16>;
    // tile slots per (segment, block group), about two workgroups per compute
    // unit in all (a workgroup keeps its weights over its tiles); at most
    // ceil(cap / 16) tiles per segment
    (void)grid;
    int tg = std::max(1, 512 / (U::OBG * NSHARD));
    tg = std::min(tg, std::max(1, (a.cap + 15) / 16));
    return launch_kernel(c, upsample_kernel<CI, CO, S, BF16>, dim3(tg * U::OBG * NSHARD), dim3(256), a);
}

hipError_t launch_upsample(const UpArgs& a, int cin, int cout, int stride, bool bf16, int grid,
                           const LaunchCtx& c) {
#define SSC_LAUNCH(CI, CO, S)                                                                               \
    if (cin == CI && cout == CO && stride == S)                                                             \
        return bf16 ? launch_up_shape<CI, CO, S, true>(a, grid, c) : launch_up_shape<CI, CO, S, false>(a, grid, c);
    SSC_UP_SHAPES(SSC_LAUNCH)
#undef SSC_LAUNCH
    return hipErrorInvalidValue;
}

size_t up_wpack_elems(int cin, int cout, int stride, bool bf16) {
    return (size_t)(bf16 ? 2 * cin : cin) * (size_t)cout * stride * stride;
}

// Layout, in 16-byte lane vectors: [chunk c][output block ob][lane l], with
// ob = (a*S + b)*NCBT + cb; lane l of block ob holds output channel
// cb*16 + l%16 of sub-cell (a, b) and the k-group l/16 of chunk c: fp32
// k = c*16 + 4*(l/16) + e (e < 4); bf16 k = c*32 + 8*(l/16) + e (e < 8) over
// the pair [W | -W].  w: [cin][cout][S][S] (fp32 values, or bf16 bits).
void pack_up_weights(const void* w, int cin, int cout, int s, bool bf16, void* dst) {
    const int ncbt = cout / 16, nob = s * s * ncbt;
    auto widx = [&](int ci, int co, int a, int b) { return (((size_t)ci * cout + co) * s + a) * s + b; };
    if (!bf16) {
        const float* src = static_cast<const float*>(w);
        float* out = static_cast<float*>(dst);
        const int nch = cin / 16;
        for (int c = 0; c < nch; ++c)
            for (int ob = 0; ob < nob; ++ob) {
                const int ab = ob / ncbt, cb = ob % ncbt;
                for (int l = 0; l < 64; ++l)
                    for (int e = 0; e < 4; ++e) {
                        const int co = cb * 16 + l % 16, ci = c * 16 + 4 * (l / 16) + e;
                        out[(((size_t)c * nob + ob) * 64 + l) * 4 + e] = src[widx(ci, co, ab / s, ab % s)];
                    }
            }
    } else {
        const uint16_t* src = static_cast<const uint16_t*>(w);
        uint16_t* out = static_cast<uint16_t*>(dst);
        const int nch = (2 * cin) / 32;
        for (int c = 0; c < nch; ++c)
            for (int ob = 0; ob < nob; ++ob) {
                const int ab = ob / ncbt, cb = ob % ncbt;
                for (int l = 0; l < 64; ++l)
                    for (int e = 0; e < 8; ++e) {
                        const int co = cb * 16 + l % 16, k = c * 32 + 8 * (l / 16) + e;
                        const int ci = k < cin ? k : k - cin;
                        uint16_t v = src[widx(ci, co, ab / s, ab % s)];
                        if (k >= cin) v ^= 0x8000u;   // -W: exact sign flip
                        out[(((size_t)c * nob + ob) * 64 + l) * 8 + e] = v;
                    }
            }
    }
}

}  // namespace ssc
