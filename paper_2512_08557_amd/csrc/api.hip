// Host side of the C ABI declared in include/sscater.h: validation, worst-case
// allocation, weight repacking and the per-stride launch sequence.
//
// Per stride, on the caller's stream, with no host synchronisation:
//   1. detect (present)  : new pillars vs canvas -> A_0 stamps, input deltas,
//                          canvas update, A_0 -> A_1 propagation;
//   2. detect (vanished) : previous list minus the new list -> same outputs,
//                          and the duplicate check of the new list;
//   3. layer l = 1..L    : contraction over A_l, Z_l update, delta epilogue,
//                          A_l -> A_{l+1} propagation;
//   4. the neck          : one upsampling launch per upsampler, when present.
// Points mode replaces 1 and 2 by the pillar queue update and the pillar
// feature net (sscater_step_points); a sparse backbone adds the active-set
// words that detect and each block's first layer keep current.
// Work sizes live in device counters; the layer kernels walk their tiles from
// the counter, so the host never waits for a count.
//
// Every change set is the set of cells stamped with the stride's epoch in a
// per-grid stamp map, and every delta row sits at its cell's position;
// bumping the epoch invalidates every set at once, so no per-stride clears are
// needed.  The output sets of the layers are also compacted into lists of
// NSHARD segments.  The two counter sets alternate between strides; the
// detect launch clears the set the next stride will use.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/sscater.h"
#include "sscater_internal.h"

using namespace ssc;

namespace {

struct LayerState {
    sscater_layer spec{};
    int Hin = 0, Win = 0, Hout = 0, Wout = 0;
    float* Z = nullptr;
    void* wpack = nullptr;
    uint32_t* stamp = nullptr;
    int32_t* list = nullptr; // NSHARD segments of Hout*Wout cells
    void* delta = nullptr;   // deltas of this layer's output, dense by cell (nullptr for the last layer)
    // sparse backbones: the output active-set words (owned by a regular
    // layer, shared with the submanifold layers of its block)
    uint64_t* memb = nullptr;
    bool sub = false;
    // wide stride-1 layers after the first: two launches, the contraction of
    // the changed input rows with all nine taps, then the tap sum
    bool split = false;
    void* wg = nullptr;      // contraction weights [9*cout][cin]
};

// One upsampler of the neck.
struct UpState {
    sscater_upsampler spec{};
    int cin = 0;
    int Hs = 0, Ws = 0;      // source grid
    int coff = 0;            // first channel in the neck map
    void* wpack = nullptr;
};

thread_local char g_hip_err[256] = "no HIP error";

int hip_fail(hipError_t e) {
    snprintf(g_hip_err, sizeof g_hip_err, "HIP error %d: %s", (int)e, hipGetErrorString(e));
    return e == hipErrorOutOfMemory ? SSCATER_E_OUT_OF_MEMORY : SSCATER_E_HIP;
}

size_t round_up(size_t n, size_t a) { return (n + a - 1) / a * a; }

int out_extent(int n, int s) { return (n + 2 - 3) / s + 1; }

}  // namespace

struct sscater {
    int device = 0;
    sscater_grid grid{};
    int L = 0;
    int batch = 1;                 // independent images of H x W cells each
    bool bf16 = false;
    int row_bytes = 0;      // bytes of one input feature row
    LayerState layers[SSCATER_MAX_LAYERS];
    // neck: upsamplers into one concatenated map on the grid Hn x Wn
    int n_ups = 0;
    UpState ups[SSCATER_MAX_UPSAMPLERS];
    int Hn = 0, Wn = 0, Cn = 0;
    float* Zn = nullptr;
    uint32_t* stamp_n = nullptr;
    float* part = nullptr;         // tap contributions of a split layer, dense by cell (shared by those layers)
    float* zero = nullptr;         // a zero row of 9 * max cout floats
    void* X = nullptr;
    uint64_t* pres = nullptr;
    uint32_t* stamp0 = nullptr;
    void* delta0 = nullptr;
    int32_t* prev[2] = {nullptr, nullptr};
    int prev_slot = 0;
    int32_t prev_count = 0;
    bool prev_dense = false;
    bool prev_sorted = true;       // the previous list is known to increase (or is empty)
    // [2 sets][nlines()][CSTRIDE], word 0 of each line a counter: per set the
    // list lengths cnt[0..L][shard], then pairs[0..L][shard][PSPREAD], then the
    // detection's |A_0| adds [shard][PSPREAD] (statistics; points mode counts
    // A_0 in cnt[0], the length of the list it builds)
    int32_t* counters = nullptr;
    long long* cum = nullptr;      // running totals, same layout as one set
    int32_t* err_host = nullptr;   // host-visible sticky error word
    int32_t* err_dev = nullptr;
    bool sparse = false;           // regular sparse + submanifold layers
    // points mode: the incremental pillar feature net in front of the layers
    bool pfn = false;
    sscater_pfn pfn_spec{};
    float inv_res = 0.f;
    float4* ring = nullptr;        // [cells][N] point queues
    uint32_t* head = nullptr;      // [cells] points removed
    uint32_t* tail = nullptr;      // [cells] points inserted
    uint32_t* scnt = nullptr;      // [window + 1][cells] points per cell of each stride slot
    int32_t* touched = nullptr;    // [window + 1][max_new_points] cells each stride slot touched
    int32_t* tcount = nullptr;     // [window + 1][CSTRIDE] their counters
    uint32_t* ins_stamp = nullptr; // [cells]
    int32_t* list0 = nullptr;      // A_0 list, NSHARD segments of cells
    float* pfn_w = nullptr;        // [C0][9]
    uint32_t epoch = 0;
    int last_set = -1;             // counter set of the last stride, -1 after create/reset
    uint32_t last_epoch = 0;       // epoch of the last stride
    long long steps = 0;
    int32_t last_pillars = 0;
    int layer_grid = 1024;
    std::vector<void*> allocs;
    // per-kernel event timing (metrics extension)
    struct ProfRec {
        int slot;
        hipEvent_t a, b;
    };
    bool prof = false;
    std::vector<hipEvent_t> ev_pool;
    size_t ev_next = 0;
    std::vector<ProfRec> prof_recs;

    int nlines() const { return (L + 1) * NSHARD * (1 + PSPREAD) + NSHARD * PSPREAD; }
    int ncnt() const { return nlines() * CSTRIDE; }
    // cells of layer l's output grid over the whole batch (l = 0: the input)
    size_t cells_of(int l) const {
        return (size_t)batch * (l == 0 ? (size_t)grid.H * grid.W : (size_t)layers[l - 1].Hout * layers[l - 1].Wout);
    }
    int32_t* cnt_ptr(int set, int l) { return set_ptr(set) + (size_t)l * NSHARD * CSTRIDE; }
    int32_t* pairs_ptr(int set, int l) {
        return set_ptr(set) + ((size_t)(L + 1) * NSHARD + (size_t)l * NSHARD * PSPREAD) * CSTRIDE;
    }
    int32_t* a0_ptr(int set) { return set_ptr(set) + (size_t)(L + 1) * NSHARD * (1 + PSPREAD) * CSTRIDE; }
    int32_t* set_ptr(int s) { return counters + (size_t)s * ncnt(); }
};

namespace {

struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) { ok = false; return; }
        if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

int dev_alloc(sscater* h, void** p, size_t bytes) {
    bytes = round_up(bytes < 256 ? 256 : bytes, 256);
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) { *p = nullptr; return hip_fail(e); }
    h->allocs.push_back(*p);
    e = hipMemset(*p, 0, bytes);
    if (e != hipSuccess) return hip_fail(e);
    return SSCATER_OK;
}

void free_all(sscater* h) {
    for (void* p : h->allocs) (void)hipFree(p);
    h->allocs.clear();
    for (hipEvent_t e : h->ev_pool) (void)hipEventDestroy(e);
    h->ev_pool.clear();
    if (h->err_host) (void)hipHostFree(h->err_host);
    h->err_host = nullptr;
}

bool pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

int check_sticky(const sscater* h) {
    return (h->err_host && __atomic_load_n(h->err_host, __ATOMIC_ACQUIRE) != 0) ? SSCATER_E_DEVICE : SSCATER_OK;
}

hipError_t prof_event(sscater* h, hipEvent_t* out) {
    if (h->ev_next == h->ev_pool.size()) {
        hipEvent_t e;
        hipError_t r = hipEventCreate(&e);
        if (r != hipSuccess) return r;
        h->ev_pool.push_back(e);
    }
    *out = h->ev_pool[h->ev_next++];
    return hipSuccess;
}

// Launch wrapper: while profiling is enabled the launch carries two events
// that its dispatch stamps at the kernel's start and end.
template <class F>
hipError_t timed_launch(sscater* h, int slot, hipStream_t s, F&& launch) {
    LaunchCtx c;
    c.stream = s;
    if (!h->prof) return launch(c);
    sscater::ProfRec r{slot, nullptr, nullptr};
    hipError_t e = prof_event(h, &r.a);
    if (e == hipSuccess) e = prof_event(h, &r.b);
    if (e != hipSuccess) return e;
    c.start = r.a;
    c.stop = r.b;
    e = launch(c);
    if (e == hipSuccess) h->prof_recs.push_back(r);
    return e;
}

PropTarget prop_target(sscater* h, int l /* consuming layer, 1..L */, int set) {
    PropTarget t{};
    const LayerState& ls = h->layers[l - 1];
    t.stride = ls.spec.stride;
    t.Hin = ls.Hin;
    t.Win = ls.Win;
    t.Hout = ls.Hout;
    t.Wout = ls.Wout;
    t.seg = (int)h->cells_of(l);
    t.stamp = ls.stamp;
    t.list = ls.list;
    t.count = h->cnt_ptr(set, l);
    t.pairs = h->pairs_ptr(set, l);
    return t;
}

// The layers and the neck of one stride, after A_0 and A_1 are built.
int run_layers(sscater* h, int set, uint32_t epoch, hipStream_t s) {
    int32_t* cnt = h->set_ptr(set);
    hipError_t e = hipSuccess;
    for (int l = 1; l <= h->L; ++l) {
        LayerState& ls = h->layers[l - 1];
        LayerArgs a{};
        a.list = ls.list;
        a.count = h->cnt_ptr(set, l);
        a.cap = (int)h->cells_of(l);
        a.stamp_in = l == 1 ? h->stamp0 : h->layers[l - 2].stamp;
        a.delta_in = l == 1 ? h->delta0 : h->layers[l - 2].delta;
        a.wpack = ls.wpack;
        a.Z = ls.Z;
        a.delta_out = ls.delta;   // allocated when a later layer or an upsampler reads it
        a.Hin = ls.Hin;
        a.Win = ls.Win;
        a.Hout = ls.Hout;
        a.Wout = ls.Wout;
        a.relu = ls.spec.relu;
        a.epoch = epoch;
        a.has_next = l < h->L;
        if (a.has_next) a.next = prop_target(h, l + 1, set);
        if (h->sparse) {
            a.memb = ls.memb;
            if (!ls.sub)      // a regular layer passes its membership changes to the next regular layer
                for (int k = l + 1; k <= h->L; ++k)
                    if (!h->layers[k - 1].sub) {
                        const LayerState& nx = h->layers[k - 1];
                        a.mnext = MembTarget{nx.memb, nx.spec.stride, nx.Hout, nx.Wout};
                        break;
                    }
        }
        if (l == h->L) {
            a.cum_src = cnt;
            a.cum_dst = h->cum;
            a.n_cum = h->nlines();
        }
        if (ls.split) {
            ContractArgs g{};
            g.list = h->layers[l - 2].list;
            g.count = h->cnt_ptr(set, l - 1);
            g.cap = (int)h->cells_of(l - 1);
            g.delta_in = a.delta_in;
            g.wg = ls.wg;
            g.part = h->part;
            e = timed_launch(h, h->L + 1 + h->n_ups + l, s, [&](const LaunchCtx& c) {
                return launch_contract(g, ls.spec.cin, ls.spec.cout, h->bf16, h->layer_grid, c);
            });
            if (e != hipSuccess) return hip_fail(e);
            a.part = h->part;
            a.zero = h->zero;
            e = timed_launch(h, 1 + l, s, [&](const LaunchCtx& c) {
                return launch_tap_sum(a, ls.spec.cout, h->bf16, h->sparse, h->layer_grid, c);
            });
        } else {
            e = timed_launch(h, 1 + l, s, [&](const LaunchCtx& c) {
                return launch_layer(a, ls.spec.cin, ls.spec.cout, ls.spec.stride, h->bf16, h->sparse, h->layer_grid,
                                    c);
            });
        }
        if (e != hipSuccess) return hip_fail(e);
    }

    // the neck: every upsampler over its source layer's change list
    for (int u = 0; u < h->n_ups; ++u) {
        const UpState& us = h->ups[u];
        const LayerState& src = h->layers[us.spec.src_layer - 1];
        UpArgs a{};
        a.list = src.list;
        a.count = h->cnt_ptr(set, us.spec.src_layer);
        a.cap = src.Hout * src.Wout;
        a.delta_src = src.delta;
        a.wpack = us.wpack;
        a.Z = h->Zn;
        a.ctot = h->Cn;
        a.coff = us.coff;
        a.stamp = h->stamp_n;
        a.Wsrc = us.Ws;
        a.epoch = epoch;
        e = timed_launch(h, h->L + 2 + u, s, [&](const LaunchCtx& c) {
            return launch_upsample(a, us.cin, us.spec.cout, us.spec.stride, h->bf16, h->layer_grid, c);
        });
        if (e != hipSuccess) return hip_fail(e);
    }
    return SSCATER_OK;
}

}  // namespace

extern "C" {

const char* sscater_strerror(int code) {
    switch (code) {
        case SSCATER_OK: return "ok";
        case SSCATER_E_INVALID_ARG: return "invalid argument";
        case SSCATER_E_OUT_OF_MEMORY: return "out of memory";
        case SSCATER_E_HIP: return g_hip_err;
        case SSCATER_E_OVERFLOW: return "pillar count exceeds max_pillars (no sampling)";
        case SSCATER_E_SCRATCH: return "grid larger than the fixed scratch of an allocation-free call (64 Mi cells)";
        case SSCATER_E_DEVICE:
            return "device-side input fault (cell index out of range, duplicate cell, or a pillar over its point "
                   "capacity)";
        default: return "unknown error";
    }
}

int sscater_create(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                   const void* const* weights, sscater_t* out) {
    return sscater_create_neck(grid, layers, n_layers, weights, nullptr, 0, nullptr, out);
}

}  // extern "C"

namespace {

int create_impl(const sscater_grid* grid, int32_t batch, const sscater_layer* layers, int32_t n_layers,
                const void* const* weights, const sscater_upsampler* ups, int32_t n_ups,
                const void* const* up_weights, sscater_t* out) {
    // ---- validation: host only, before any HIP call ----
    if (!grid || !layers || !weights || !out) return SSCATER_E_INVALID_ARG;
    if (batch < 1 || (batch > 1 && n_ups > 0)) return SSCATER_E_INVALID_ARG;
    if (n_ups < 0 || n_ups > SSCATER_MAX_UPSAMPLERS || (n_ups > 0 && (!ups || !up_weights))) return SSCATER_E_INVALID_ARG;
    *out = nullptr;
    if (grid->H <= 0 || grid->W <= 0 || grid->C0 <= 0 || grid->max_pillars < 0) return SSCATER_E_INVALID_ARG;
    if (grid->H >= 32768 || grid->W >= 32768) return SSCATER_E_INVALID_ARG;   // cell coordinates fit 15 bits
    if (grid->dtype != SSCATER_F32 && grid->dtype != SSCATER_BF16) return SSCATER_E_INVALID_ARG;
    if (n_layers < 1 || n_layers > SSCATER_MAX_LAYERS) return SSCATER_E_INVALID_ARG;
    const bool bf16 = grid->dtype == SSCATER_BF16;
    const long long cells0 = (long long)grid->H * grid->W * batch;
    if (cells0 > (1LL << 30)) return SSCATER_E_INVALID_ARG;
    const int row_bytes = grid->C0 * (bf16 ? 2 : 4);
    if (!pow2(row_bytes) || row_bytes < 16 || row_bytes > 1024) return SSCATER_E_INVALID_ARG;
    {
        int H = grid->H, W = grid->W, C = grid->C0;
        for (int l = 0; l < n_layers; ++l) {
            const sscater_layer& s = layers[l];
            if (s.k != 3 || s.pad != 1 || (s.stride != 1 && s.stride != 2) || (s.relu != 0 && s.relu != 1))
                return SSCATER_E_INVALID_ARG;
            if (s.cin != C || !layer_supported(s.cin, s.cout, s.stride, bf16)) return SSCATER_E_INVALID_ARG;
            if (!weights[l]) return SSCATER_E_INVALID_ARG;
            H = out_extent(H, s.stride);
            W = out_extent(W, s.stride);
            C = s.cout;
        }
    }
    // upsamplers: a backbone layer's output, kernel = stride in {1, 2, 4}, all
    // onto one grid, concatenated
    int Hn = 0, Wn = 0;
    for (int u = 0; u < n_ups; ++u) {
        const sscater_upsampler& up = ups[u];
        if (up.src_layer < 1 || up.src_layer > n_layers || (up.relu != 0 && up.relu != 1) || !up_weights[u])
            return SSCATER_E_INVALID_ARG;
        int H = grid->H, W = grid->W;
        for (int l = 0; l < up.src_layer; ++l) {
            H = out_extent(H, layers[l].stride);
            W = out_extent(W, layers[l].stride);
        }
        const int cin = layers[up.src_layer - 1].cout;
        if (!upsample_supported(cin, up.cout, up.stride)) return SSCATER_E_INVALID_ARG;
        if (u == 0) {
            Hn = H * up.stride;
            Wn = W * up.stride;
        } else if (H * up.stride != Hn || W * up.stride != Wn) {
            return SSCATER_E_INVALID_ARG;
        }
    }

    sscater* h = new (std::nothrow) sscater();
    if (!h) return SSCATER_E_OUT_OF_MEMORY;
    h->grid = *grid;
    h->batch = batch;
    h->L = n_layers;
    h->bf16 = bf16;
    h->row_bytes = row_bytes;
    // layer launches: 1024 workgroups per image, at most 4096 (a batch of
    // images carries that many more tiles per launch; measured on four
    // 1024x1024 images: 4096 workgroups 196 us per stride against 202 us
    // with 1024); SSCATER_LAYER_GRID overrides it
    h->layer_grid = (int)std::min<long long>(4096, 1024LL * batch);
    if (const char* g = getenv("SSCATER_LAYER_GRID")) {
        const int v = atoi(g);
        if (v >= 32 && v <= 65536) h->layer_grid = v & ~31;
    }
    hipError_t he = hipGetDevice(&h->device);
    if (he != hipSuccess) {
        delete h;
        return hip_fail(he);
    }

    int rc = SSCATER_OK;
    const size_t esz = bf16 ? 2 : 4;
    // SSCATER_FUSED_WIDE=1 keeps every wide stride-1 layer in the one-launch
    // output-stationary kernel (for comparing the two forms)
    const char* fw = getenv("SSCATER_FUSED_WIDE");
    const bool split_wide = !(fw && atoi(fw) != 0);
    const size_t cells = (size_t)cells0;
#define SSC_TRY(expr)                 \
    do {                              \
        rc = (expr);                  \
        if (rc != SSCATER_OK) goto fail; \
    } while (0)
    SSC_TRY(dev_alloc(h, &h->X, cells * row_bytes));
    SSC_TRY(dev_alloc(h, (void**)&h->pres, cells * 8));
    SSC_TRY(dev_alloc(h, (void**)&h->stamp0, cells * 4));
    // input deltas dense by cell: fp32 rows or bf16 [new | old] pairs
    SSC_TRY(dev_alloc(h, &h->delta0, cells * (size_t)(bf16 ? 2 * row_bytes : row_bytes)));
    SSC_TRY(dev_alloc(h, (void**)&h->prev[0], (size_t)grid->max_pillars * 4));
    SSC_TRY(dev_alloc(h, (void**)&h->prev[1], (size_t)grid->max_pillars * 4));
    SSC_TRY(dev_alloc(h, (void**)&h->counters, (size_t)2 * h->ncnt() * 4));
    SSC_TRY(dev_alloc(h, (void**)&h->cum, (size_t)h->ncnt() * 8));
    {
        int H = grid->H, W = grid->W;
        size_t part_bytes = 0, zero_bytes = 0;
        for (int l = 0; l < n_layers; ++l) {
            LayerState& ls = h->layers[l];
            ls.spec = layers[l];
            ls.Hin = H;
            ls.Win = W;
            ls.Hout = out_extent(H, ls.spec.stride);
            ls.Wout = out_extent(W, ls.spec.stride);
            const size_t oc = (size_t)batch * ls.Hout * ls.Wout;
            SSC_TRY(dev_alloc(h, (void**)&ls.Z, oc * ls.spec.cout * 4));
            SSC_TRY(dev_alloc(h, (void**)&ls.stamp, oc * 4));
            SSC_TRY(dev_alloc(h, (void**)&ls.list, oc * 4 * NSHARD));
            bool feeds_up = false;
            for (int u = 0; u < n_ups; ++u) feeds_up = feeds_up || ups[u].src_layer == l + 1;
            if (l + 1 < n_layers || feeds_up) SSC_TRY(dev_alloc(h, &ls.delta, oc * ls.spec.cout * 4));
            // the first layer's input list is not built (detection propagates
            // A_0 straight into A_1), so it always takes the one-launch kernel
            ls.split = l > 0 && split_wide && contract_supported(ls.spec.cin, ls.spec.cout, ls.spec.stride, bf16);
            if (ls.split) {
                const size_t wn = (size_t)9 * ls.spec.cout * ls.spec.cin;
                std::vector<unsigned char> packed(wn * esz);
                pack_contract_weights(weights[l], ls.spec.cin, ls.spec.cout, bf16, packed.data());
                SSC_TRY(dev_alloc(h, &ls.wg, wn * esz));
                he = hipMemcpy(ls.wg, packed.data(), wn * esz, hipMemcpyHostToDevice);
                if (he != hipSuccess) { rc = hip_fail(he); goto fail; }
                part_bytes = std::max(part_bytes, (size_t)batch * H * W * 9 * ls.spec.cout * 4);
                zero_bytes = std::max(zero_bytes, (size_t)9 * ls.spec.cout * 4);
            } else {
                const size_t wn = wpack_elems(ls.spec.cin, ls.spec.cout, bf16);
                std::vector<unsigned char> packed(wn * esz);
                pack_weights(weights[l], ls.spec.cin, ls.spec.cout, bf16, packed.data());
                SSC_TRY(dev_alloc(h, &ls.wpack, wn * esz));
                he = hipMemcpy(ls.wpack, packed.data(), wn * esz, hipMemcpyHostToDevice);
                if (he != hipSuccess) { rc = hip_fail(he); goto fail; }
            }
            H = ls.Hout;
            W = ls.Wout;
        }
        if (part_bytes) {
            SSC_TRY(dev_alloc(h, (void**)&h->part, part_bytes));
            SSC_TRY(dev_alloc(h, (void**)&h->zero, zero_bytes));
        }
    }
    if (n_ups > 0) {
        h->n_ups = n_ups;
        h->Hn = Hn;
        h->Wn = Wn;
        for (int u = 0; u < n_ups; ++u) {
            UpState& us = h->ups[u];
            us.spec = ups[u];
            const LayerState& src = h->layers[ups[u].src_layer - 1];
            us.cin = src.spec.cout;
            us.Hs = src.Hout;
            us.Ws = src.Wout;
            us.coff = h->Cn;
            h->Cn += ups[u].cout;
            const size_t wn = up_wpack_elems(us.cin, ups[u].cout, ups[u].stride, bf16);
            std::vector<unsigned char> packed(wn * esz);
            pack_up_weights(up_weights[u], us.cin, ups[u].cout, ups[u].stride, bf16, packed.data());
            SSC_TRY(dev_alloc(h, &us.wpack, wn * esz));
            he = hipMemcpy(us.wpack, packed.data(), wn * esz, hipMemcpyHostToDevice);
            if (he != hipSuccess) { rc = hip_fail(he); goto fail; }
        }
        SSC_TRY(dev_alloc(h, (void**)&h->Zn, (size_t)Hn * Wn * h->Cn * 4));
        SSC_TRY(dev_alloc(h, (void**)&h->stamp_n, (size_t)Hn * Wn * 4));
    }
    he = hipHostMalloc((void**)&h->err_host, 256, hipHostMallocMapped | hipHostMallocCoherent);
    if (he != hipSuccess) { h->err_host = nullptr; rc = hip_fail(he); goto fail; }
    *h->err_host = 0;
    he = hipHostGetDevicePointer((void**)&h->err_dev, h->err_host, 0);
    if (he != hipSuccess) { rc = hip_fail(he); goto fail; }
    he = hipDeviceSynchronize();
    if (he != hipSuccess) { rc = hip_fail(he); goto fail; }
#undef SSC_TRY
    h->epoch = 0;
    *out = h;
    return SSCATER_OK;
fail:
    free_all(h);
    delete h;
    return rc;
}

}  // namespace

extern "C" {

int sscater_create_neck(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                        const void* const* weights, const sscater_upsampler* ups, int32_t n_ups,
                        const void* const* up_weights, sscater_t* out) {
    return create_impl(grid, 1, layers, n_layers, weights, ups, n_ups, up_weights, out);
}

int sscater_create_batched(const sscater_grid* grid, int32_t batch, const sscater_layer* layers, int32_t n_layers,
                           const void* const* weights, sscater_t* out) {
    return create_impl(grid, batch, layers, n_layers, weights, nullptr, 0, nullptr, out);
}

// sorted: the caller's cell indices increase strictly (sscater_step_sorted)
static int step_impl(sscater_t h, const sscater_pillars* pl, void* stream, bool sorted) {
    if (!h || !pl || h->pfn) return SSCATER_E_INVALID_ARG;
    if (int rc = check_sticky(h)) return rc;
    const long long cells = (long long)h->cells_of(0);
    // NULL idx with count == H*W is dense mode; NULL idx with count 0 is an empty stride
    const bool dense = pl->idx == nullptr && pl->count != 0;
    if (dense && h->sparse) return SSCATER_E_INVALID_ARG;   // the pillar set is part of a sparse input
    if (dense) {
        if (pl->count != cells || !pl->feats) return SSCATER_E_INVALID_ARG;
    } else {
        if (pl->count < 0) return SSCATER_E_INVALID_ARG;
        if (pl->count > h->grid.max_pillars) return SSCATER_E_OVERFLOW;
        if (pl->count > 0 && !pl->feats) return SSCATER_E_INVALID_ARG;
    }
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);

    const uint32_t epoch = ++h->epoch;
    const int set = (int)(epoch & 1u);
    int32_t* cnt = h->set_ptr(set);
    const int cur_slot = h->prev_slot ^ 1;

    DetectArgs d{};
    d.idx = pl->idx;
    d.feats = pl->feats;
    d.count = pl->count;
    d.prev = nullptr;
    d.prev_out = dense ? nullptr : h->prev[cur_slot];
    d.X = h->X;
    d.pres = h->pres;
    d.stamp0 = h->stamp0;
    d.count0 = h->a0_ptr(set);
    d.delta0 = h->delta0;
    d.zero_ptr = h->set_ptr(set ^ 1);
    d.zero_n = h->nlines();
    d.HW = (int32_t)cells;
    d.epoch = epoch;
    d.err = h->err_dev;
    d.next = prop_target(h, 1, set);
    if (h->sparse) {
        const LayerState& l1 = h->layers[0];
        d.memb = MembTarget{l1.memb, l1.spec.stride, l1.Hout, l1.Wout};
    }
    // Sorted lists: one launch that merges the new list with the previous
    // one chunk by chunk; it needs the previous list sorted too, so a stride
    // after a dense one or after an sscater_step (whose list may come in any
    // order) takes the two passes, which then check the order of this one.
    d.sorted = sorted && !dense ? 1 : 0;
    const bool one_launch = sorted && !dense && !h->prev_dense && h->prev_sorted;
    hipError_t e = hipSuccess;
    if (one_launch) {
        DetectArgs m = d;
        m.prev = h->prev[h->prev_slot];
        m.prev_count = h->prev_count;
        e = timed_launch(h, 0, s, [&](const LaunchCtx& c) { return launch_detect_sorted(m, h->row_bytes, h->bf16, c); });
    } else {
        e = timed_launch(h, 0, s, [&](const LaunchCtx& c) { return launch_detect_present(d, h->row_bytes, h->bf16, c); });
    }
    if (e != hipSuccess) return hip_fail(e);

    // vanished cells of the previous list, and the ownership check of the
    // new list's presence words (pillar mode only: dense input has no
    // duplicates)
    if (!one_launch && !dense && (h->prev_dense || h->prev_count > 0 || pl->count > 0)) {
        DetectArgs v = d;
        v.prev = h->prev_dense ? nullptr : h->prev[h->prev_slot];
        v.count = h->prev_dense ? (int32_t)cells : h->prev_count;
        v.chk_idx = pl->count > 0 ? pl->idx : nullptr;
        v.chk_count = pl->count;
        v.prev_out = nullptr;
        v.zero_ptr = nullptr;
        v.zero_n = 0;
        e = timed_launch(h, 1, s, [&](const LaunchCtx& c) { return launch_detect_vanished(v, h->row_bytes, h->bf16, c); });
        if (e != hipSuccess) return hip_fail(e);
    }

    if (int rc = run_layers(h, set, epoch, s)) return rc;

    if (!dense) {
        h->prev_slot = cur_slot;
        h->prev_count = pl->count;
        h->prev_dense = false;
        h->prev_sorted = sorted;
    } else {
        h->prev_count = 0;
        h->prev_dense = true;
    }
    h->last_set = set;
    h->last_epoch = epoch;
    h->steps += 1;
    h->last_pillars = pl->count;
    return SSCATER_OK;
}

int sscater_step(sscater_t h, const sscater_pillars* pl, void* stream) { return step_impl(h, pl, stream, false); }

int sscater_step_sorted(sscater_t h, const sscater_pillars* pl, void* stream) {
    return step_impl(h, pl, stream, true);
}

int sscater_create_pfn(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                       const void* const* weights, const sscater_pfn* pfn, const float* pfn_weights,
                       sscater_t* out) {
    if (!grid || !pfn || !pfn_weights || !out) return SSCATER_E_INVALID_ARG;
    *out = nullptr;
    const sscater_pfn& p = *pfn;
    if (!(p.res > 0.f) || !std::isfinite(p.res) || !std::isfinite(p.x_min) || !std::isfinite(p.y_min) ||
        p.max_points < 1 || p.max_points > 128 || p.window < 1 || p.window > 64 || p.max_new_points < 0 ||
        p.max_new_points > (1 << 24) || grid->C0 < 1 || grid->C0 > 64)
        return SSCATER_E_INVALID_ARG;
    sscater_t h = nullptr;
    int rc = sscater_create_neck(grid, layers, n_layers, weights, nullptr, 0, nullptr, &h);
    if (rc != SSCATER_OK) return rc;
    DeviceGuard dg(h->device);
    if (!dg.ok) {
        sscater_destroy(h);
        return hip_fail(hipGetLastError());
    }
    const size_t cells = (size_t)grid->H * grid->W;
    const size_t slots = (size_t)p.window + 1;
    const size_t per_slot = (size_t)std::max(p.max_new_points, 1);
    hipError_t he = hipSuccess;
    h->pfn = true;
    h->pfn_spec = p;
    h->inv_res = 1.0f / p.res;
    if ((rc = dev_alloc(h, (void**)&h->ring, cells * (size_t)p.max_points * sizeof(float4))) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->head, cells * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->tail, cells * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->scnt, slots * cells * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->touched, slots * per_slot * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->tcount, slots * CSTRIDE * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->ins_stamp, cells * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->list0, (size_t)NSHARD * cells * 4)) != SSCATER_OK ||
        (rc = dev_alloc(h, (void**)&h->pfn_w, (size_t)grid->C0 * 9 * 4)) != SSCATER_OK) {
        sscater_destroy(h);
        return rc;
    }
    he = hipMemcpy(h->pfn_w, pfn_weights, (size_t)grid->C0 * 9 * 4, hipMemcpyHostToDevice);
    if (he == hipSuccess) he = hipDeviceSynchronize();
    if (he != hipSuccess) {
        rc = hip_fail(he);
        sscater_destroy(h);
        return rc;
    }
    *out = h;
    return SSCATER_OK;
}

int sscater_step_points(sscater_t h, const float* points, int32_t n_points, void* stream) {
    if (!h || !h->pfn || n_points < 0 || (n_points > 0 && !points)) return SSCATER_E_INVALID_ARG;
    if (n_points > h->pfn_spec.max_new_points) return SSCATER_E_OVERFLOW;
    if (int rc = check_sticky(h)) return rc;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    const sscater_pfn& p = h->pfn_spec;
    const int cells = h->grid.H * h->grid.W;
    const uint32_t epoch = ++h->epoch;
    const int set = (int)(epoch & 1u);
    // stride slots: this stride inserts into slot steps % (window + 1); the
    // stride that leaves the window (steps - window) used slot (steps + 1) % (window + 1)
    const int slots = p.window + 1;
    const int ins = (int)(h->steps % slots), pop = (int)((h->steps + 1) % slots);
    const size_t per_slot = (size_t)std::max(p.max_new_points, 1);

    PillarArgs u{};
    u.points = reinterpret_cast<const float4*>(points);
    u.n_points = n_points;
    u.x_min = p.x_min;
    u.y_min = p.y_min;
    u.inv_res = h->inv_res;
    u.H = h->grid.H;
    u.W = h->grid.W;
    u.N = p.max_points;
    u.ring = h->ring;
    u.head = h->head;
    u.tail = h->tail;
    u.scnt_ins = h->scnt + (size_t)ins * cells;
    u.scnt_pop = h->scnt + (size_t)pop * cells;
    u.touched_ins = h->touched + (size_t)ins * per_slot;
    u.tcount_ins = h->tcount + (size_t)ins * CSTRIDE;
    u.touched_pop = h->touched + (size_t)pop * per_slot;
    u.tcount_pop = h->tcount + (size_t)pop * CSTRIDE;
    u.ins_stamp = h->ins_stamp;
    u.stamp0 = h->stamp0;
    u.list0 = h->list0;
    u.count0 = h->cnt_ptr(set, 0);
    u.zero_ptr = h->set_ptr(set ^ 1);
    u.zero_n = h->nlines();
    u.epoch = epoch;
    // the leaving stride touched at most max_new_points cells
    u.n_pop_blocks = std::max(1, std::min(64, (p.max_new_points + 255) / 256));
    const int ins_blocks = std::max(1, std::min(256, (n_points + 255) / 256));
    hipError_t e = timed_launch(h, 0, s, [&](const LaunchCtx& c) { return launch_pillar_update(u, ins_blocks, c); });
    if (e != hipSuccess) return hip_fail(e);

    PfnArgs f{};
    f.list0 = h->list0;
    f.count0 = h->cnt_ptr(set, 0);
    f.cap0 = cells;
    f.ring = h->ring;
    f.head = h->head;
    f.tail = h->tail;
    f.N = p.max_points;
    f.w = h->pfn_w;
    f.C0 = h->grid.C0;
    f.W = h->grid.W;
    f.x_min = p.x_min;
    f.y_min = p.y_min;
    f.res = p.res;
    f.X = h->X;
    f.delta0 = h->delta0;
    f.tcount_clear = h->tcount + (size_t)pop * CSTRIDE;   // the next stride inserts into this slot
    f.err = h->err_dev;
    f.epoch = epoch;
    f.next = prop_target(h, 1, set);
    // |A_0| <= the leaving stride's cells + this stride's points; one wavefront per pillar
    const long long bound = (long long)p.max_new_points + n_points;
    const int pfn_blocks = (int)std::max(1LL, std::min(1024LL, (bound + 3) / 4));
    e = timed_launch(h, 1, s, [&](const LaunchCtx& c) { return launch_pfn(f, h->bf16, pfn_blocks, c); });
    if (e != hipSuccess) return hip_fail(e);

    if (int rc = run_layers(h, set, epoch, s)) return rc;
    h->last_set = set;
    h->last_epoch = epoch;
    h->steps += 1;
    h->last_pillars = n_points;
    return SSCATER_OK;
}

int sscater_create_sparse(const sscater_grid* grid, const sscater_layer* layers, int32_t n_layers,
                          const void* const* weights, const int32_t* submanifold, sscater_t* out) {
    if (!grid || !layers || !submanifold || !out || n_layers < 1 || n_layers > SSCATER_MAX_LAYERS)
        return SSCATER_E_INVALID_ARG;
    *out = nullptr;
    if (submanifold[0] != 0) return SSCATER_E_INVALID_ARG;   // a sparse stack starts with a regular layer
    for (int l = 0; l < n_layers; ++l)
        if ((submanifold[l] != 0 && submanifold[l] != 1) || (submanifold[l] == 1 && layers[l].stride != 1))
            return SSCATER_E_INVALID_ARG;
    sscater_t h = nullptr;
    int rc = sscater_create_neck(grid, layers, n_layers, weights, nullptr, 0, nullptr, &h);
    if (rc != SSCATER_OK) return rc;
    DeviceGuard dg(h->device);
    if (!dg.ok) {
        sscater_destroy(h);
        return hip_fail(hipGetLastError());
    }
    for (int l = 0; l < n_layers; ++l) {
        LayerState& ls = h->layers[l];
        ls.sub = submanifold[l] == 1;
        if (ls.sub) {
            ls.memb = h->layers[l - 1].memb;
        } else if ((rc = dev_alloc(h, (void**)&ls.memb, h->cells_of(l + 1) * 8)) != SSCATER_OK) {
            sscater_destroy(h);
            return rc;
        }
    }
    h->sparse = true;
    *out = h;
    return SSCATER_OK;
}

int sscater_read(sscater_t h, int32_t layer, void* dst, size_t dst_bytes, void* stream) {
    if (!h || !dst || layer < 0 || layer > h->L + (h->n_ups > 0 ? 1 : 0)) return SSCATER_E_INVALID_ARG;
    if (int rc = check_sticky(h)) return rc;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t esz = h->bf16 ? 2 : 4;
    if (layer == 0) {
        const size_t need = h->cells_of(0) * h->row_bytes;
        if (dst_bytes < need) return SSCATER_E_INVALID_ARG;
        hipError_t e = hipMemcpyAsync(dst, h->X, need, hipMemcpyDeviceToDevice, s);
        return e == hipSuccess ? SSCATER_OK : hip_fail(e);
    }
    if (layer == h->L + 1) {   // the neck map, each upsampler's phi over its channels
        const long long cells = (long long)h->Hn * h->Wn;
        if (dst_bytes < (size_t)cells * h->Cn * esz) return SSCATER_E_INVALID_ARG;
        for (int u = 0; u < h->n_ups; ++u) {
            const UpState& us = h->ups[u];
            hipError_t e = launch_read_slice(h->Zn, dst, cells, h->Cn, us.coff, us.spec.cout, us.spec.relu, h->bf16, s);
            if (e != hipSuccess) return hip_fail(e);
        }
        return SSCATER_OK;
    }
    const LayerState& ls = h->layers[layer - 1];
    const long long n = (long long)h->cells_of(layer) * ls.spec.cout;
    if (dst_bytes < (size_t)n * esz) return SSCATER_E_INVALID_ARG;
    hipError_t e = h->sparse ? launch_read_masked(ls.Z, dst, (long long)h->cells_of(layer), ls.spec.cout, ls.memb,
                                                  ls.spec.relu, h->bf16, s)
                             : launch_read(ls.Z, dst, n, ls.spec.relu, h->bf16, s);
    return e == hipSuccess ? SSCATER_OK : hip_fail(e);
}

int sscater_reset(sscater_t h, void* stream) {
    if (!h) return SSCATER_E_INVALID_ARG;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    // The library drains the stream before clearing the host-visible error
    // word, so a fault of a stride still in flight cannot survive the reset.
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e);
    const size_t cells = h->cells_of(0);
    e = launch_fill_zero(h->X, round_up(cells * h->row_bytes, 256), s);
    for (int l = 0; l < h->L && e == hipSuccess; ++l) {
        const LayerState& ls = h->layers[l];
        e = launch_fill_zero(ls.Z, round_up(h->cells_of(l + 1) * ls.spec.cout * 4, 256), s);
    }
    if (e == hipSuccess && h->Zn) e = launch_fill_zero(h->Zn, round_up((size_t)h->Hn * h->Wn * h->Cn * 4, 256), s);
    if (e == hipSuccess) e = launch_fill_zero(h->counters, round_up((size_t)2 * h->ncnt() * 4, 256), s);
    if (e == hipSuccess) e = launch_fill_zero(h->cum, round_up((size_t)h->ncnt() * 8, 256), s);
    for (int l = 0; l < h->L && e == hipSuccess && h->sparse; ++l) {
        const LayerState& ls = h->layers[l];
        if (!ls.sub) e = launch_fill_zero(ls.memb, round_up(h->cells_of(l + 1) * 8, 256), s);
    }
    if (e == hipSuccess && h->pfn) {
        const size_t slots = (size_t)h->pfn_spec.window + 1;
        e = launch_fill_zero(h->head, round_up(cells * 4, 256), s);
        if (e == hipSuccess) e = launch_fill_zero(h->tail, round_up(cells * 4, 256), s);
        if (e == hipSuccess) e = launch_fill_zero(h->scnt, round_up(slots * cells * 4, 256), s);
        if (e == hipSuccess) e = launch_fill_zero(h->tcount, round_up(slots * CSTRIDE * 4, 256), s);
    }
    if (e != hipSuccess) return hip_fail(e);
    ++h->epoch;   // every stamp becomes stale
    h->prev_count = 0;
    h->prev_dense = false;
    h->prev_sorted = true;
    h->last_set = -1;
    h->steps = 0;
    h->last_pillars = 0;
    __atomic_store_n(h->err_host, 0, __ATOMIC_RELEASE);
    return SSCATER_OK;
}

int sscater_destroy(sscater_t h) {
    if (!h) return SSCATER_E_INVALID_ARG;
    {
        DeviceGuard dg(h->device);
        free_all(h);
    }
    delete h;
    return SSCATER_OK;
}

}  // extern "C"

namespace ssc {

int report_hip_error(hipError_t e) { return hip_fail(e); }

int changed_source(const sscater* h, int layer, ChangedSource* out) {
    if (!h || !out || layer < 0 || layer > h->L + (h->n_ups > 0 ? 1 : 0)) return SSCATER_E_INVALID_ARG;
    if (int rc = check_sticky(h)) return rc;
    ChangedSource c;
    c.device = h->device;
    c.have = h->last_set >= 0;
    c.epoch = h->last_epoch;
    if (layer == 0) {
        c.stamp = h->stamp0;
        c.cells = (long long)h->cells_of(0);
    } else if (layer == h->L + 1) {
        c.stamp = h->stamp_n;
        c.cells = (long long)h->Hn * h->Wn;
    } else {
        c.stamp = h->layers[layer - 1].stamp;
        c.cells = (long long)h->cells_of(layer);
        if (h->sparse) c.memb = h->layers[layer - 1].memb;
    }
    *out = c;
    return SSCATER_OK;
}

}  // namespace ssc

extern "C" {

int sscater_changed(sscater_t h, int32_t layer, int32_t* dst, int32_t cap, int32_t* count_host, void* stream) {
    if (!h || !count_host || layer < 0 || layer > h->L + (h->n_ups > 0 ? 1 : 0) || cap < 0 || (cap > 0 && !dst))
        return SSCATER_E_INVALID_ARG;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e);
    if (int rc = check_sticky(h)) return rc;
    if (h->last_set < 0) {
        *count_host = 0;
        return SSCATER_OK;
    }
    std::vector<int32_t> buf;
    if (layer == 0 || layer == h->L + 1) {
        // A_0 and the neck's set: the cells stamped with the last stride's epoch
        const int cells = layer == 0 ? (int)h->cells_of(0) : h->Hn * h->Wn;
        std::vector<uint32_t> st((size_t)cells);
        e = hipMemcpy(st.data(), layer == 0 ? h->stamp0 : h->stamp_n, st.size() * 4, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e);
        for (int q = 0; q < cells; ++q)
            if (st[(size_t)q] == h->last_epoch) buf.push_back(q);
    } else {
        int32_t cnt[NSHARD * CSTRIDE];
        e = hipMemcpy(cnt, h->cnt_ptr(h->last_set, layer), sizeof cnt, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e);
        // the list segments; a segment never holds more entries than its grid has cells
        const LayerState& ls = h->layers[layer - 1];
        const int cap_cells = (int)h->cells_of(layer);
        for (int k = 0; k < NSHARD; ++k) {
            const int m = std::min(std::max(cnt[k * CSTRIDE], 0), cap_cells);
            if (m == 0) continue;
            const size_t at = buf.size();
            buf.resize(at + (size_t)m);
            e = hipMemcpy(buf.data() + at, ls.list + (size_t)k * cap_cells, (size_t)m * 4, hipMemcpyDeviceToHost);
            if (e != hipSuccess) return hip_fail(e);
        }
    }
    if (h->sparse && layer >= 1 && layer <= h->L && !buf.empty()) {
        // a sparse layer's changed sites: its work list minus the sites that
        // are active neither now nor in the previous stride
        const LayerState& ls = h->layers[layer - 1];
        std::vector<uint64_t> mw(h->cells_of(layer));
        e = hipMemcpy(mw.data(), ls.memb, mw.size() * 8, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e);
        const uint64_t ep = h->last_epoch & 0x7FFFFFFFu;
        size_t k = 0;
        for (int32_t q : buf) {
            const uint64_t w = mw[(size_t)q];
            const bool now = (uint32_t)w != 0u;
            const bool prev = (w >> 33) == ep ? ((w >> 32) & 1ull) != 0ull : now;
            if (now || prev) buf[k++] = q;
        }
        buf.resize(k);
    }
    const int32_t n = (int32_t)buf.size();
    *count_host = n;
    if (n == 0) return SSCATER_OK;
    std::sort(buf.begin(), buf.end());
    std::memcpy(dst, buf.data(), (size_t)std::min(n, cap) * 4);
    return SSCATER_OK;
}

int sscater_stats(sscater_t h, sscater_stats_t* out, void* stream) {
    if (!h || !out) return SSCATER_E_INVALID_ARG;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e);
    std::memset(out, 0, sizeof *out);
    const int L = h->L;
    out->n_layers = L;
    out->steps = h->steps;
    out->pillars = h->last_pillars;
    std::vector<int32_t> c((size_t)h->ncnt(), 0);
    std::vector<long long> t((size_t)h->ncnt(), 0);
    if (h->last_set >= 0) {
        e = hipMemcpy(c.data(), h->set_ptr(h->last_set), c.size() * 4, hipMemcpyDeviceToHost);
        if (e != hipSuccess) return hip_fail(e);
    }
    e = hipMemcpy(t.data(), h->cum, t.size() * 8, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e);
    std::vector<long long> act(L + 1, 0), prs(L + 1, 0);
    for (int l = 0; l <= L; ++l) {
        long long a_c = 0, p_c = 0, a_t = 0, p_t = 0;
        for (int k = 0; k < NSHARD; ++k) {
            a_c += c[((size_t)l * NSHARD + k) * CSTRIDE];
            a_t += t[((size_t)l * NSHARD + k) * CSTRIDE];
            if (l == 0)
                for (int x = 0; x < PSPREAD; ++x) {
                    const size_t line = (size_t)(L + 1) * NSHARD * (1 + PSPREAD) + (size_t)k * PSPREAD + x;
                    a_c += c[line * CSTRIDE];
                    a_t += t[line * CSTRIDE];
                }
            for (int x = 0; x < PSPREAD; ++x) {
                const size_t line = (size_t)(L + 1) * NSHARD + ((size_t)l * NSHARD + k) * PSPREAD + x;
                p_c += c[line * CSTRIDE];
                p_t += t[line * CSTRIDE];
            }
        }
        act[l] = a_c;
        prs[l] = p_c;
        out->active[l] = (int32_t)a_c;
        out->pairs[l] = (int32_t)p_c;
        out->active_total[l] = a_t;
        out->pairs_total[l] = p_t;
    }
    // algorithmic flops and HBM bytes of the last stride (the method's own work)
    const double e_in = h->bf16 ? 2.0 : 4.0;        // stored feature element
    const double e_d = 4.0;                          // delta element (fp32, or bf16 pair)
    const double P = (double)h->last_pillars, C0 = (double)h->grid.C0;
    double flops = 0.0;
    double bytes = P * (4.0 + C0 * e_in)             // new pillar list
                   + P * C0 * e_in                   // canvas compare gather
                   + (double)act[0] * C0 * (e_in + e_d);  // canvas write + input deltas
    for (int l = 1; l <= L; ++l) {
        const sscater_layer& sp = h->layers[l - 1].spec;
        const double a_in = (double)act[l - 1], a_out = (double)act[l], pairs = (double)prs[l];
        flops += 2.0 * sp.cin * sp.cout * pairs;
        bytes += a_in * sp.cin * e_d                 // input deltas
                 + a_out * sp.cout * 8.0             // Z read + write
                 + (l < L ? a_out * sp.cout * e_d : 0.0)   // emitted deltas
                 + 9.0 * sp.cin * sp.cout * e_in     // weights
                 + 8.0 * (a_in + a_out);             // lists and stamps
    }
    out->n_ups = h->n_ups;
    for (int u = 0; u < h->n_ups; ++u) {
        const UpState& us = h->ups[u];
        const long long s2 = (long long)us.spec.stride * us.spec.stride;
        const double a_src = (double)act[us.spec.src_layer];
        out->up_pairs[u] = act[us.spec.src_layer] * s2;
        flops += 2.0 * us.cin * us.spec.cout * a_src * (double)s2;
        bytes += a_src * us.cin * e_d                              // source deltas
                 + a_src * (double)s2 * us.spec.cout * 8.0         // neck Z read + write
                 + (double)us.cin * us.spec.cout * s2 * e_in       // weights
                 + a_src * (4.0 + (double)s2 * 4.0);               // list entries, stamps
    }
    out->flops = flops;
    out->bytes = bytes;
    return check_sticky(h);
}

int sscater_profile(sscater_t h, int32_t enable) {
    if (!h) return SSCATER_E_INVALID_ARG;
    h->prof = enable != 0;
    return SSCATER_OK;
}

int sscater_profile_read(sscater_t h, double* ms, int64_t* launches, int32_t n, void* stream) {
    if (!h || !ms || !launches || n < 2 * h->L + 2 + h->n_ups) return SSCATER_E_INVALID_ARG;
    DeviceGuard dg(h->device);
    if (!dg.ok) return hip_fail(hipGetLastError());
    hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e);
    for (int i = 0; i < n; ++i) {
        ms[i] = 0.0;
        launches[i] = 0;
    }
    for (const auto& r : h->prof_recs) {
        float t = 0.f;
        e = hipEventElapsedTime(&t, r.a, r.b);
        if (e != hipSuccess) return hip_fail(e);
        ms[r.slot] += t;
        launches[r.slot] += 1;
    }
    h->prof_recs.clear();
    h->ev_next = 0;
    return SSCATER_OK;
}

}  // extern "C"
