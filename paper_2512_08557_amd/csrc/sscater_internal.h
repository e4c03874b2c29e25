// Internal definitions shared by the library's HIP translation units.
// Kernel arguments are plain structs passed by value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssc {

// Change-list propagation target: the next layer's grid and its list state.
// A cell q of the target grid belongs to the current stride's list when
// stamp[q] == epoch; map[q] = (epoch << 32) | position of q in `list`.
struct PropTarget {
    int stride;           // stride of the layer that consumes this list
    int Hin, Win;         // grid the changed cells live in
    int Hout, Wout;       // grid of the target list
    uint32_t* stamp;      // [Hout*Wout]
    uint64_t* map;        // [Hout*Wout]
    int32_t* list;        // [Hout*Wout]
    int32_t* count;       // device counter of the target list
    int32_t* pairs;       // device counter of (input, output) pairs of the consuming layer
};

// Changed-cell detection on the input canvas.
struct DetectArgs {
    const int32_t* idx;   // pillar cell indices (nullptr: dense mode, cell = i)
    const void* feats;    // pillar feature rows (present mode)
    int32_t count;        // rows to examine
    const int32_t* prev;  // previous stride's cell list (vanish mode; nullptr: all cells)
    int32_t* prev_out;    // copy of this stride's cell list (present mode, may be nullptr)
    void* X;              // persistent canvas [H0*W0][row bytes]
    uint32_t* pres;       // presence stamps [H0*W0]
    uint64_t* map0;       // (epoch << 32) | row in A_0
    int32_t* list0;       // A_0
    int32_t* count0;      // |A_0| counter
    void* delta0;         // packed input deltas in A_0 order
    int32_t* zero_ptr;    // counters to clear for the next stride (may be nullptr)
    int32_t zero_n;
    int32_t HW;
    uint32_t epoch;
    int32_t* err;         // sticky error flags (host-visible memory)
    PropTarget next;
};

// One convolution layer: contraction of the packed input deltas with the
// weights, update of the persistent pre-activation map, activation delta
// epilogue and propagation of the change list to the next layer.
struct LayerArgs {
    const int32_t* list;      // A_l (cells of the output grid)
    const int32_t* count;     // |A_l|
    int cap;                  // capacity of `list` (cells of the output grid)
    const uint64_t* map_in;   // index map of A_{l-1} on the input grid
    const void* delta_in;     // packed deltas of layer l-1 in A_{l-1} order
    const void* wpack;        // weights repacked for the MFMA operand layout
    float* Z;                 // persistent pre-activation map [Hout*Wout][cout]
    void* delta_out;          // packed deltas of layer l in A_l order (nullptr: last layer)
    int Hin, Win, Hout, Wout;
    int relu;
    uint32_t epoch;
    int has_next;
    PropTarget next;
    // running totals, folded in by the last layer of a stride
    const int32_t* cum_src;   // this stride's counters [n_cum]
    long long* cum_dst;       // totals [n_cum]
    int n_cum;
};

enum ErrBits { ERR_INDEX_RANGE = 1, ERR_DUPLICATE = 2 };

// Host-side launchers (defined in the kernel translation units).
hipError_t launch_detect_present(const DetectArgs& a, int row_bytes, bool bf16, hipStream_t s);
hipError_t launch_detect_vanished(const DetectArgs& a, int row_bytes, bool bf16, hipStream_t s);
bool layer_supported(int cin, int cout, int stride, bool bf16);
hipError_t launch_layer(const LayerArgs& a, int cin, int cout, int stride, bool bf16, int grid,
                        hipStream_t s);
hipError_t launch_read(const float* Z, void* dst, long long n, int relu, bool bf16, hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
size_t wpack_elems(int cin, int cout, bool bf16);
// Repack OIHW weights (fp32 values, or bf16 bit patterns) into the layout the
// layer kernel reads; dst holds wpack_elems() elements of 4 (fp32) or 2 (bf16) bytes.
void pack_weights(const void* w_oihw, int cin, int cout, bool bf16, void* dst);

}  // namespace ssc
