// Internal definitions shared by the library's HIP translation units.
// Kernel arguments are plain structs passed by value.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

struct sscater;   // the handle (api.hip)

namespace ssc {

// Change sets.  A cell q of a grid belongs to the current stride's set when
// stamp[q] == epoch; bumping the epoch empties every set at once.
// Delta rows are stored at their cell's position (a consumer checks the stamp
// before it gathers a row, so stale rows are never read).  The output sets of
// the layers are also compacted into lists, the work lists of the layer
// kernels.  A list is NSHARD segments, each with its own counter, filled by
// the workgroups b with b % NSHARD == shard: on gfx950 every device-scope
// atomic executes beyond the per-XCD L2, and appends of all workgroups to one
// counter queue on that one address.  Workgroup b runs on XCD b % 8.
constexpr int NSHARD = 2;
// Distance between the counters of two segments (in int32): one 128-byte line
// each, since atomics on different words of one line still queue together.
constexpr int CSTRIDE = 32;
// The pairs counter of a (layer, segment) is spread over PSPREAD lines, one per
// XCD of the adding workgroup, and summed by the host: every wavefront that
// appends to a list also adds its pairs, and on one line those adds queue
// behind each other on the list builders' critical path.
constexpr int PSPREAD = 8;
static_assert((PSPREAD & (PSPREAD - 1)) == 0, "PSPREAD indexes by blockIdx.x & (PSPREAD - 1)");

// Change-list propagation target: the next layer's grid and its list state.
// A handle may hold a batch of independent images: cell index
// b * (H * W) + r * W + c; every neighbourhood stays inside its image.
struct PropTarget {
    int stride;           // stride of the layer that consumes this list
    int Hin, Win;         // image the changed cells live in
    int Hout, Wout;       // image of the target list
    int seg;              // cells of one list segment: batch * Hout * Wout
    uint32_t* stamp;      // [Hout*Wout]
    int32_t* list;        // NSHARD segments of Hout*Wout entries
    int32_t* count;       // segment lengths, segment k at count[k * CSTRIDE]
    int32_t* pairs;       // (input, output) pairs of the consuming layer: segment k,
                          // XCD x at pairs[(k * PSPREAD + x) * CSTRIDE]
};

// Sparse backbones (regular sparse and submanifold convolutions): every
// layer's output sites carry an active-set word,
//   bits 0..31  number of active input sites in the site's receptive field
//               (the site is active while it is not zero),
//   bit 32      whether the site was active at the end of the previous stride,
//   bits 33..63 the epoch (mod 2^31) of the word's last change,
// so both the current and the previous active set are read from one word.
// A submanifold layer shares the word array of the regular layer that starts
// its block (it keeps the active set).  Membership changes go one level down:
// pillar toggles update the first regular layer's words, a regular layer's
// kernel updates the next regular layer's words for its sites that changed.
struct MembTarget {
    uint64_t* memb;       // words of the next regular layer's output grid (nullptr: none)
    int stride;           // that layer's stride
    int Hout, Wout;       // its output grid (its input grid is the source grid)
};

// Changed-cell detection on the input canvas.
struct DetectArgs {
    const int32_t* idx;   // pillar cell indices (nullptr: dense mode, cell = i)
    const void* feats;    // pillar feature rows (present mode)
    int32_t count;        // rows to examine
    const int32_t* prev;  // previous stride's cell list (vanish and sorted modes; nullptr: all cells)
    int32_t prev_count;   // its length (sorted mode)
    int32_t sorted;       // the new list was passed as increasing strictly: checked in the present pass
    int32_t* prev_out;    // copy of this stride's cell list (present mode, may be nullptr)
    void* X;              // persistent canvas [H0*W0][row bytes]
    uint64_t* pres;       // presence words [H0*W0]: (epoch << 32) | row of the pillar in this stride's list
    const int32_t* chk_idx;   // vanish mode: this stride's pillar list, checked for duplicate cells (may be nullptr)
    int32_t chk_count;
    uint32_t* stamp0;     // change stamps of the input grid [H0*W0]
    int32_t* count0;      // |A_0| (statistics only): segment k, XCD x at count0[(k * PSPREAD + x) * CSTRIDE]
    void* delta0;         // input deltas, dense by cell [H0*W0][4*C0 bytes]
    int32_t* zero_ptr;    // counters to clear for the next stride (may be nullptr)
    int32_t zero_n;       // their lines (word 0 of each CSTRIDE line is the counter)
    int32_t HW;
    uint32_t epoch;
    int32_t* err;         // sticky error flags (host-visible memory)
    PropTarget next;
    MembTarget memb;      // sparse backbones: the first layer's active-set words
};

// One convolution layer: contraction of the input deltas with the weights,
// update of the persistent pre-activation map, activation delta epilogue and
// propagation of the change list to the next layer.
struct LayerArgs {
    const int32_t* list;        // A_l: NSHARD segments of `cap` cells of the output grid
    const int32_t* count;       // segment lengths, segment k at count[k * CSTRIDE]
    int cap;                    // capacity of a segment (cells of the output grid)
    const uint32_t* stamp_in;   // change stamps of the input grid [Hin*Win]
    const void* delta_in;       // input deltas, dense by cell [Hin*Win][4*cin bytes]
    const void* wpack;          // weights repacked for the MFMA operand layout
    float* Z;                   // persistent pre-activation map [Hout*Wout][cout]
    void* delta_out;            // output deltas, dense by cell (nullptr: last layer)
    int Hin, Win, Hout, Wout;
    int relu;
    uint32_t epoch;
    int has_next;
    PropTarget next;
    // sparse backbones: this layer's output active-set words, and where a
    // regular layer sends its sites' membership changes
    const uint64_t* memb;
    MembTarget mnext;
    // running totals, folded in by the last layer of a stride
    const int32_t* cum_src;     // this stride's counters, word 0 of n_cum CSTRIDE lines
    long long* cum_dst;         // totals, the same layout
    int n_cum;
    // layers contracted in two launches (tap_sum_kernel): the tap
    // contributions of the changed input cells, dense by cell
    // [Hin*Win][9][cout] fp32, and a zero row of 9*cout floats that stands
    // in for an unchanged input
    const float* part;
    const float* zero;
};

// The scatter form of Eq. 2 for one stride-1 layer: every changed input row
// times the weights of all nine taps, [|A_{l-1}| x cin] x [cin x 9*cout].
struct ContractArgs {
    const int32_t* list;        // A_{l-1}: NSHARD segments of `cap` cells of the input grid
    const int32_t* count;       // segment lengths, segment k at count[k * CSTRIDE]
    int cap;
    const void* delta_in;       // input deltas, dense by cell [Hin*Win][4*cin bytes]
    const void* wg;             // weights [9*cout][cin] (fp32, or bf16 values), row tap*cout + co
    float* part;                // tap contributions, dense by cell [Hin*Win][9*cout]
};

// One upsampler of the neck: transposed convolution (kernel = stride) of a
// backbone layer's output deltas into the persistent concatenated neck map.
struct UpArgs {
    const int32_t* list;        // the source layer's change list: NSHARD segments of `cap` cells
    const int32_t* count;       // segment lengths, segment k at count[k * CSTRIDE]
    int cap;                    // cells of the source grid
    const void* delta_src;      // source deltas, dense by cell [Hsrc*Wsrc][4*cin bytes]
    const void* wpack;          // weights repacked for the MFMA operand layout
    float* Z;                   // neck pre-activation map [Hn*Wn][ctot]
    int ctot, coff;             // channels of the neck map, first channel of this upsampler
    uint32_t* stamp;            // change stamps of the neck grid [Hn*Wn]
    int Wsrc;                   // width of the source grid (Wn = stride * Wsrc)
    uint32_t epoch;
};

// Pillar point queues of the incremental pillar feature net: every cell holds
// a ring of N points; tail counts the points ever inserted, head those
// removed, so the live points are ring positions head..tail-1 (mod N).  The
// points of one stride leave the window together, `window` strides later, so
// per-stride slots (window + 1 of them) keep, per cell, how many points that
// stride inserted and the list of cells it touched.
struct PillarArgs {
    const float4* points;       // this stride's points (x, y, z, intensity)
    int n_points;
    float x_min, y_min, inv_res;
    int H, W, N;
    float4* ring;               // [H*W][N]
    uint32_t* head;             // [H*W]
    uint32_t* tail;             // [H*W]
    uint32_t* scnt_ins;         // [H*W] points per cell of this stride's slot
    uint32_t* scnt_pop;         // [H*W] ... of the slot of the stride leaving the window
    int32_t* touched_ins;       // cells first touched by this stride, and their counter
    int32_t* tcount_ins;
    const int32_t* touched_pop; // cells the leaving stride touched, and their count
    const int32_t* tcount_pop;
    uint32_t* ins_stamp;        // [H*W] epoch of a cell's last insertion
    uint32_t* stamp0;           // [H*W] A_0 stamps
    int32_t* list0;             // A_0 list, NSHARD segments of H*W
    int32_t* count0;            // its counters, segment k at [k * CSTRIDE]
    int32_t* zero_ptr;          // counter set of the next stride, cleared here
    int zero_n;                 // its lines
    uint32_t epoch;
    int n_pop_blocks;           // workgroups [0, n_pop_blocks) remove, the others insert
};

// The pillar feature net over A_0: decoration, pointwise linear layer, ReLU
// and max over each changed pillar's points; the canvas update, the input
// deltas and A_0 -> A_1 propagation as in change detection.
struct PfnArgs {
    const int32_t* list0;
    const int32_t* count0;
    int cap0;                   // cells per list segment
    const float4* ring;
    const uint32_t* head;
    const uint32_t* tail;
    int N;
    const float* w;             // [C0][9]
    int C0, W;
    float x_min, y_min, res;
    void* X;                    // canvas [H*W][C0] (grid dtype)
    void* delta0;               // input deltas dense by cell
    int32_t* tcount_clear;      // counter of the next stride's insertion slot, cleared here
    int32_t* err;
    uint32_t epoch;
    PropTarget next;
};

// ERR_UNSORTED: a list passed as sorted does not increase.
enum ErrBits { ERR_INDEX_RANGE = 1, ERR_DUPLICATE = 2, ERR_PILLAR_FULL = 4, ERR_UNSORTED = 8 };

// What a layer's change list is made of, for the device-side list: the cells
// q of the layer's grid with stamp[q] == epoch, restricted for a sparse layer
// to the sites active now or in the previous stride.
struct ChangedSource {
    const uint32_t* stamp = nullptr;
    const uint64_t* memb = nullptr;   // sparse layers only
    uint32_t epoch = 0;
    long long cells = 0;              // cells of the grid (whole batch)
    int device = 0;
    bool have = false;                // a stride has run since create / reset
};
// SSCATER_OK, SSCATER_E_INVALID_ARG (null handle, layer out of range) or
// SSCATER_E_DEVICE (sticky device fault).
int changed_source(const sscater* h, int layer, ChangedSource* out);
// Record a HIP error for sscater_strerror; returns the matching error code.
int report_hip_error(hipError_t e);

// Where a launch goes: its stream and, while kernel timing is on, two events
// that the dispatch packet itself stamps when the kernel starts and ends
// (hipExtLaunchKernel), so no separate marker packets sit between kernels.
struct LaunchCtx {
    hipStream_t stream = nullptr;
    hipEvent_t start = nullptr, stop = nullptr;
};

template <class K, class... A>
inline hipError_t launch_kernel(const LaunchCtx& c, K kernel, dim3 grid, dim3 block, const A&... args) {
    if (c.start) hipExtLaunchKernelGGL(kernel, grid, block, 0, c.stream, c.start, c.stop, 0, args...);
    else hipLaunchKernelGGL(kernel, grid, block, 0, c.stream, args...);
    return hipGetLastError();
}

// Host-side launchers (defined in the kernel translation units).
hipError_t launch_detect_present(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c);
hipError_t launch_detect_vanished(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c);
hipError_t launch_detect_sorted(const DetectArgs& a, int row_bytes, bool bf16, const LaunchCtx& c);
bool layer_supported(int cin, int cout, int stride, bool bf16);
hipError_t launch_layer(const LayerArgs& a, int cin, int cout, int stride, bool bf16, bool sparse, int grid,
                        const LaunchCtx& c);
hipError_t launch_read(const float* Z, void* dst, long long n, int relu, bool bf16, hipStream_t s);
// phi(Z) with the sites outside the active set (sparse backbones) zeroed.
hipError_t launch_read_masked(const float* Z, void* dst, long long cells, int cout, const uint64_t* memb, int relu,
                              bool bf16, hipStream_t s);
// phi of channels [coff, coff + cout) of a [cells][ctot] map into the same
// channels of a [cells][ctot] destination.
hipError_t launch_read_slice(const float* Z, void* dst, long long cells, int ctot, int coff, int cout, int relu,
                             bool bf16, hipStream_t s);
// Wide stride-1 layers: the contraction of the changed input rows with all
// nine taps into `part`, then the output-stationary sum of the tap
// contributions with the Z update, the delta epilogue and the propagation.
bool contract_supported(int cin, int cout, int stride, bool bf16);
hipError_t launch_contract(const ContractArgs& a, int cin, int cout, bool bf16, int grid, const LaunchCtx& c);
hipError_t launch_tap_sum(const LayerArgs& a, int cout, bool bf16, bool sparse, int grid, const LaunchCtx& c);
// [9*cout][cin] contraction weights from OIHW (fp32 values, or bf16 bits).
void pack_contract_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst);
bool upsample_supported(int cin, int cout, int stride);
hipError_t launch_upsample(const UpArgs& a, int cin, int cout, int stride, bool bf16, int grid,
                           const LaunchCtx& c);
size_t up_wpack_elems(int cin, int cout, int stride, bool bf16);
// Repack [cin][cout][S][S] transposed-conv weights (fp32 values, or bf16 bits)
// into the layout the upsampling kernel reads.
void pack_up_weights(const void* w, int cin, int cout, int stride, bool bf16, void* dst);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_pillar_update(const PillarArgs& a, int insert_blocks, const LaunchCtx& c);
hipError_t launch_pfn(const PfnArgs& a, bool bf16, int blocks, const LaunchCtx& c);
size_t wpack_elems(int cin, int cout, bool bf16);
// Repack OIHW weights (fp32 values, or bf16 bit patterns) into the layout the
// layer kernel reads; dst holds wpack_elems() elements of 4 (fp32) or 2 (bf16) bytes.
void pack_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst);

}  // namespace ssc
