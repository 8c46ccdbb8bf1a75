// C ABI of libbcpnn (declared in include/bcpnn.h): argument checks, state ownership, launches.
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "bcpnn_internal.h"

using bcpnn::Geometry;

namespace {

constexpr int32_t kMaxOutMcu = 1024;     // softmax segment held in LDS by the support kernel
constexpr int32_t kMaxInHcu = 49152;     // mask column held in LDS by the swap kernel
constexpr int32_t kMaxSwaps = 256;
// operand sets: one group filling, up to two being swept
constexpr int kSets = 3 * bcpnn::kMaxSweepBatches;
// 32 x 32 blocks of Pij per CU up to which the sweep runs with one workgroup per CU
constexpr int64_t kSmallSweepBlocksPerCu = 64;

thread_local std::string g_error;

// Scratch of bcpnn_structural_update_static: the MI scores ([in_hcu][out_hcu] fp64) and the
// per-hidden-HCU swap counts of the update in flight.  Each GPU the library runs on holds its
// own copy until the process ends; every such call on a GPU shares it.  Host code uses the
// device address resolved per device (static_scratch), never the array's name.
constexpr size_t kStaticScratchBytes = 32u << 20;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on device `dev`, which must be current; resolved once per
// device.
hipError_t static_scratch(int dev, void** out) {
    *out = nullptr;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

bcpnn_status fail(bcpnn_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return st;
}

}  // namespace

struct bcpnn_layer {
    bcpnn_config cfg;
    Geometry g;
    hipStream_t stream = nullptr;        // the caller's stream
    hipStream_t side = nullptr;          // the layer's own stream for the silent-trace sweep
    int drop_bits = 0;
    int32_t max_active = 0;              // largest active count of a hidden HCU (swaps keep it)
    float* pi[2] = {nullptr, nullptr};   // the trace kernel reads one and writes the other
    float* pj[2] = {nullptr, nullptr};
    int cur = 0;
    float* pij = nullptr;
    float* w = nullptr;
    float* b = nullptr;
    uint8_t* mask = nullptr;             // [in_hcu][out_hcu]
    int32_t* act_list = nullptr;         // [out_hcu][in_hcu], ascending active input HCUs
    int32_t* act_count = nullptr;        // [out_hcu]
    int32_t* swap_count = nullptr;       // [out_hcu]
    double* mi = nullptr;                // [in_hcu][out_hcu]
    int32_t* pair_error = nullptr;       // input check of complement pairs (device flag)
    int32_t pair_error_host = 0;         // its copy, read with the waits of the waiting calls
    // Split batch operands of the joint-trace contraction, kSets sets used in turn.  The silent
    // elements of Pij take the updates of up to kMaxSweepBatches consecutive batches in one
    // sweep on the side stream, which reads those batches' sets while later batches proceed.
    bcpnn::TraceOperands ops[kSets] = {};
    int ops_cur = 0;
    int64_t set_sweep[kSets];            // sweep (sequence number) that frees the set, or -1
    struct Pending { int set; int32_t B; float c1, c2; };
    Pending pend[bcpnn::kMaxSweepBatches];
    int n_pend = 0;                      // batches whose silent updates are not yet enqueued
    hipEvent_t sweep_ready = nullptr;    // the pending batches' operands are written
    hipEvent_t sweep_done[kSets] = {};   // ring of sweep completion events
    int64_t n_sweeps = 0;                // sweeps enqueued; sweep k records sweep_done[k % kSets]
    int64_t waited = -1;                 // the caller's stream already waits for sweeps <= this
    bool full_mask = false;              // no silent block: no sweeps
    int64_t sweep_wgs = 0;               // sweep launch: one workgroup per CU, or -1 (tiles)
    bool mi_valid = false;
    bool failed = false;
    void* scratch = nullptr;             // this device's static scratch (resolved at create)
    int32_t profile_every = 0;           // 0: off; n: every n-th launch of a kernel is timed
    int clock_khz = 0;                   // rate of the device clock the stamps read
    struct KernelTimer {                 // the timed launches of one kernel
        std::vector<std::pair<hipEvent_t, hipEvent_t>> events;   // event pairs around them
        std::vector<unsigned long long*> stamps;  // or device chunks of stamp slots
        size_t used = 0;
        int64_t launches = 0;
    };
    KernelTimer timers[5];               // indexed by bcpnn_kernel
};

#define HIP_TRY(layer, expr)                                                             \
    do {                                                                                 \
        hipError_t e_ = (expr);                                                          \
        if (e_ != hipSuccess) {                                                          \
            (layer)->failed = true;                                                      \
            return fail(BCPNN_EDEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));  \
        }                                                                                \
    } while (0)

namespace {

const char* check_config(const bcpnn_config* c) {
    if (!c) return "config is NULL";
    if (c->in_hcu <= 0 || c->in_mcu <= 0 || c->out_hcu <= 0 || c->out_mcu <= 0)
        return "HCU and MCU counts must be positive";
    if (c->out_mcu > kMaxOutMcu) return "out_mcu exceeds 1024";
    if (c->in_hcu > kMaxInHcu) return "in_hcu exceeds 49152";
    const int64_t n_in = (int64_t)c->in_hcu * c->in_mcu, n_out = (int64_t)c->out_hcu * c->out_mcu;
    if (n_in > (1ll << 31) - 1 || n_out > (1ll << 31) - 1) return "unit counts exceed 2^31 - 1";
    if ((n_in + 63) / 64 > 65535) return "N_in exceeds 65535 * 64";
    if (n_out > (1ll << 22)) return "N_out exceeds 2^22";      // a 64-row Pij tile < 2^30 bytes
    if (c->max_batch <= 0 || c->max_batch > (1 << 20)) return "max_batch must lie in [1, 2^20]";
    // every launch grid stays below 2^32 work-items
    if (n_in * n_out > (1ll << 35)) return "N_in * N_out exceeds 2^35";
    if ((int64_t)c->in_hcu * c->out_hcu > (1ll << 26)) return "in_hcu * out_hcu exceeds 2^26";
    if ((int64_t)((c->max_batch + 15) / 16) * c->out_hcu > (1ll << 23))
        return "ceil(max_batch / 16) * out_hcu exceeds 2^23";
    if (!(c->alpha > 0.0f && c->alpha <= 1.0f)) return "alpha must lie in (0, 1]";
    if (c->n_cycles < 1) return "n_cycles must be >= 1";
    if (!(c->gain >= 0.0f) || !isfinite(c->gain)) return "gain must be finite and >= 0";
    if (!isfinite(c->bias_gain)) return "bias_gain must be finite";
    if (!(c->eps >= FLT_MIN) || !isfinite(c->eps)) return "eps must be a finite normal float > 0";
    if (!isfinite(c->pi_init) || !isfinite(c->pj_init) || c->pi_init > 1.0f || c->pj_init > 1.0f)
        return "pi_init / pj_init must be finite and <= 1";
    if (!isfinite(c->init_noise) || c->init_noise < 0.0f) return "init_noise must be finite and >= 0";
    if (c->n_swaps < 0 || c->n_swaps > kMaxSwaps) return "n_swaps must lie in [0, 256]";
    if (c->storage != BCPNN_STORE_F32 && c->storage != BCPNN_STORE_BF16 &&
        c->storage != BCPNN_STORE_M10)
        return "unknown storage format";
    if (c->complement_pairs != 0 && c->complement_pairs != 1)
        return "complement_pairs must be 0 or 1";
    if (c->complement_pairs && c->in_mcu != 2) return "complement_pairs needs in_mcu == 2";
    return nullptr;
}

// Checks a host mask and builds the per-hidden-HCU active lists; max_active receives the
// largest count.
const char* build_active_lists(const bcpnn_config& c, const uint8_t* mask,
                               std::vector<int32_t>& list, std::vector<int32_t>& count,
                               int32_t& max_active) {
    list.assign((size_t)c.out_hcu * c.in_hcu, 0);
    count.assign((size_t)c.out_hcu, 0);
    for (int32_t hi = 0; hi < c.in_hcu; ++hi)
        for (int32_t hj = 0; hj < c.out_hcu; ++hj) {
            const uint8_t m = mask ? mask[(size_t)hi * c.out_hcu + hj] : 1;
            if (m > 1) return "mask entries must be 0 or 1";
            if (m) list[(size_t)hj * c.in_hcu + count[hj]++] = hi;
        }
    max_active = 0;
    for (int32_t hj = 0; hj < c.out_hcu; ++hj) {
        if (count[hj] == 0) return "every hidden HCU needs at least one active input HCU";
        if (count[hj] > max_active) max_active = count[hj];
    }
    if ((int64_t)max_active * c.in_mcu > bcpnn::kMaxActiveUnits)
        return "a hidden HCU has more than 12288 active input units (active HCUs * in_mcu)";
    const Geometry g{c.in_hcu, c.in_mcu, c.out_hcu, c.out_mcu, (int64_t)c.in_hcu * c.in_mcu,
                     (int64_t)c.out_hcu * c.out_mcu};
    // (with complement pairs, the larger of the two launch shapes)
    const int mode = c.complement_pairs ? bcpnn::kPairsSplit : bcpnn::kUnpaired;
    if (bcpnn::trace_active_workgroups(g, max_active, mode) >= (1ll << 24))
        return "the active-block trace launch would exceed 2^24 workgroups "
               "(out_hcu * ceil(active units / 32) * ceil(out_mcu / 128) too large)";
    return nullptr;
}

void free_layer(bcpnn_layer* L) {
    if (!L) return;
    void* bufs[] = {L->pi[0], L->pi[1], L->pj[0], L->pj[1], L->pij, L->w, L->b, L->mask,
                    L->act_list, L->act_count, L->swap_count, L->mi, L->pair_error};
    for (void* p : bufs)
        if (p) (void)hipFree(p);
    for (int k = 0; k < kSets; ++k) {
        void* ob[] = {L->ops[k].x_hi, L->ops[k].x_lo, L->ops[k].t_hi, L->ops[k].t_lo,
                      L->ops[k].x_sum, L->ops[k].t_sum};
        for (void* p : ob)
            if (p) (void)hipFree(p);
        if (L->sweep_done[k]) (void)hipEventDestroy(L->sweep_done[k]);
    }
    if (L->sweep_ready) (void)hipEventDestroy(L->sweep_ready);
    if (L->side) (void)hipStreamDestroy(L->side);
    for (auto& tm : L->timers) {
        for (auto& ev : tm.events) {
            (void)hipEventDestroy(ev.first);
            (void)hipEventDestroy(ev.second);
        }
        for (unsigned long long* p : tm.stamps) (void)hipFree(p);
    }
    delete L;
}

// Event pair for this launch of kernel k when profiling selects it (every profile_every-th
// launch), else nulls.
hipError_t timer_events(bcpnn_layer* L, int k, hipEvent_t* start, hipEvent_t* stop) {
    *start = *stop = nullptr;
    bcpnn_layer::KernelTimer& tm = L->timers[k];
    if (L->profile_every <= 0 || tm.launches++ % L->profile_every != 0) return hipSuccess;
    if (tm.used == tm.events.size()) {
        std::pair<hipEvent_t, hipEvent_t> p{nullptr, nullptr};
        hipError_t e = hipEventCreate(&p.first);
        if (e == hipSuccess) e = hipEventCreate(&p.second);
        if (e != hipSuccess) {
            if (p.first) (void)hipEventDestroy(p.first);
            return e;
        }
        tm.events.push_back(p);
    }
    *start = tm.events[tm.used].first;
    *stop = tm.events[tm.used].second;
    ++tm.used;
    return hipSuccess;
}

// The kernels of train_batch on the caller's stream (support, active blocks) are short next to
// the passage of an event through a busy stream, so they time themselves: each timed launch
// gets a slot of start and end words that its workgroups stamp with the device clock; its
// duration is the first start to the last end.
constexpr size_t kStampChunk = 256;      // slots per device allocation
constexpr size_t kSlotWords = 2 * bcpnn::kStampLanes;

bool stamped(int k) { return k == BCPNN_KERNEL_SUPPORT || k == BCPNN_KERNEL_ACTIVE; }

// Host image of blank slots: the starts at the largest value (atomic min), the ends at 0
// (atomic max).
const unsigned long long* blank_stamps() {
    static const std::vector<unsigned long long> v = [] {
        std::vector<unsigned long long> b(kSlotWords * kStampChunk, 0ull);
        for (size_t i = 0; i < kStampChunk; ++i)
            for (int l = 0; l < bcpnn::kStampLanes; ++l) b[kSlotWords * i + l] = ~0ull;
        return b;
    }();
    return v.data();
}

// Stamp slot for this launch of kernel k when profiling selects it, else null.  A slot is
// blank when handed out: chunks are blanked when allocated and their used slots when read.
hipError_t timer_stamp(bcpnn_layer* L, int k, unsigned long long** stamp) {
    *stamp = nullptr;
    bcpnn_layer::KernelTimer& tm = L->timers[k];
    if (L->profile_every <= 0 || tm.launches++ % L->profile_every != 0) return hipSuccess;
    const size_t chunk = tm.used / kStampChunk;
    if (chunk == tm.stamps.size()) {
        const size_t bytes = kSlotWords * kStampChunk * sizeof(unsigned long long);
        unsigned long long* p = nullptr;
        hipError_t e = hipMalloc(&p, bytes);
        if (e == hipSuccess) e = hipMemcpy(p, blank_stamps(), bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            if (p) (void)hipFree(p);
            return e;
        }
        tm.stamps.push_back(p);
    }
    *stamp = tm.stamps[chunk] + kSlotWords * (tm.used % kStampChunk);
    ++tm.used;
    return hipSuccess;
}

// Sum (ms) of the durations in the used stamp slots of a timer, which are blanked again.  The
// launches must be complete.  A slot no workgroup stamped (an empty grid) counts as zero.
hipError_t read_stamps(bcpnn_layer* L, bcpnn_layer::KernelTimer& tm, double* sum_ms) {
    *sum_ms = 0.0;
    std::vector<unsigned long long> h(kSlotWords * kStampChunk);
    for (size_t c = 0; c * kStampChunk < tm.used; ++c) {
        const size_t n = std::min(kStampChunk, tm.used - c * kStampChunk);
        const size_t bytes = kSlotWords * n * sizeof(unsigned long long);
        hipError_t e = hipMemcpy(h.data(), tm.stamps[c], bytes, hipMemcpyDeviceToHost);
        if (e == hipSuccess) e = hipMemcpy(tm.stamps[c], blank_stamps(), bytes, hipMemcpyHostToDevice);
        if (e != hipSuccess) return e;
        for (size_t i = 0; i < n; ++i) {
            const unsigned long long* s = h.data() + kSlotWords * i;
            unsigned long long t0 = ~0ull, t1 = 0;
            for (int l = 0; l < bcpnn::kStampLanes; ++l) {
                t0 = std::min(t0, s[l]);
                t1 = std::max(t1, s[bcpnn::kStampLanes + l]);
            }
            if (t1 > t0) *sum_ms += (double)(t1 - t0) / L->clock_khz;
        }
    }
    return hipSuccess;
}

hipError_t wait_sweep(bcpnn_layer* L, int64_t seq);

// Enqueues the silent-element sweep of the pending batches, after the caller's stream has
// written their operands.  join: the caller's stream is about to wait for it (a state access or
// a structural update), so the sweep runs there, after every earlier sweep, over the whole
// machine.
hipError_t launch_pending_sweep(bcpnn_layer* L, bool join = false, bool timed = true) {
    if (L->n_pend == 0) return hipSuccess;
    bcpnn::SweepArgs a{};
    for (int t = 0; t < L->n_pend; ++t) {
        const bcpnn::TraceOperands& o = L->ops[L->pend[t].set];
        a.bt[t] = bcpnn::SweepBatch{o.x_hi, o.x_lo, o.t_hi, o.t_lo, o.t_sum,
                                    (L->pend[t].B + 15) / 16, L->pend[t].c1, L->pend[t].c2};
    }
    a.n_batches = L->n_pend;
    a.n_ks = L->ops[0].n_ks;
    a.paired = L->ops[0].paired;
    a.pij = L->pij;
    a.mask = L->mask;
    a.drop_bits = L->drop_bits;
    hipEvent_t t0 = nullptr, t1 = nullptr;
    hipError_t e = timed ? timer_events(L, BCPNN_KERNEL_SWEEP, &t0, &t1) : hipSuccess;
    if (e != hipSuccess) return e;
    // A small layer's sweep overlaps the next batches on the side stream, one workgroup per CU.
    // A large layer's tiled sweep runs in order on the caller's stream: it fills the machine,
    // and beside it the support and active-block kernels lose more time than the overlap gains.
    const bool in_order = join || L->sweep_wgs < 0;
    hipStream_t s = in_order ? L->stream : L->side;
    const int64_t wgs = in_order && L->sweep_wgs > 0 ? 0 : L->sweep_wgs;
    if (in_order && L->n_sweeps > 0) e = wait_sweep(L, L->n_sweeps - 1);   // earlier sweeps
    const int64_t seq = L->n_sweeps++;
    const int slot = (int)(seq % kSets);
    if (e == hipSuccess && s != L->stream) {
        e = hipEventRecord(L->sweep_ready, L->stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(s, L->sweep_ready, 0);
    }
    if (e == hipSuccess) e = bcpnn::launch_trace_sweep(s, L->g, a, wgs, t0, t1);
    if (e == hipSuccess) e = hipEventRecord(L->sweep_done[slot], s);
    if (e != hipSuccess) return e;
    for (int t = 0; t < L->n_pend; ++t) L->set_sweep[L->pend[t].set] = seq;
    L->n_pend = 0;
    return hipSuccess;
}

// Makes the caller's stream wait for sweep seq and every earlier one (they run in order).
hipError_t wait_sweep(bcpnn_layer* L, int64_t seq) {
    if (seq <= L->waited) return hipSuccess;
    const hipError_t e = hipStreamWaitEvent(L->stream, L->sweep_done[seq % kSets], 0);
    if (e == hipSuccess) L->waited = seq;
    return e;
}

// Applies the pending silent updates and makes the caller's stream wait for the last sweep:
// every Pij is then current in stream order.  timed = false never creates profiling events.
hipError_t join_side(bcpnn_layer* L, bool timed = true) {
    hipError_t e = launch_pending_sweep(L, true, timed);
    if (e == hipSuccess && L->n_sweeps > 0) e = wait_sweep(L, L->n_sweeps - 1);
    return e;
}

// Enqueues the read of the device's input check (complement pairs) ahead of a wait.
hipError_t read_input_check(bcpnn_layer* L) {
    if (!L->cfg.complement_pairs) return hipSuccess;
    return hipMemcpyAsync(&L->pair_error_host, L->pair_error, sizeof(int32_t),
                          hipMemcpyDeviceToHost, L->stream);
}

// After the wait: EINPUT (and the layer marked failed) if a training input broke the pair
// property the layer was configured with.
bcpnn_status input_check_result(bcpnn_layer* L) {
    if (!L->pair_error_host) return BCPNN_OK;
    L->failed = true;
    return fail(BCPNN_EINPUT, "complement_pairs is set but a training batch held an input pair "
                              "(x_2p, x_2p+1) that does not add up to 1: the joint traces of the "
                              "second units are not those of the inputs");
}

bool mask_is_full(const bcpnn_config& c, const std::vector<int32_t>& count) {
    for (int32_t v : count)
        if (v != c.in_hcu) return false;
    return true;
}

bcpnn_status usable(const bcpnn_layer* L) {
    if (!L) return fail(BCPNN_EINVAL, "layer is NULL");
    if (L->failed) return fail(BCPNN_ESTATE, "layer failed earlier: %s", g_error.c_str());
    return BCPNN_OK;
}

bcpnn_status check_batch(const bcpnn_layer* L, int32_t B) {
    if (B < 1 || B > L->cfg.max_batch)
        return fail(BCPNN_EINVAL, "batch %d outside [1, %d]", B, L->cfg.max_batch);
    return BCPNN_OK;
}

// Caller buffers are read and written with 16-byte vector accesses.
bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

template <typename T>
hipError_t dalloc(T** p, size_t n) {
    return hipMalloc((void**)p, n * sizeof(T) ? n * sizeof(T) : 1);
}

}  // namespace

extern "C" {

void bcpnn_config_default(bcpnn_config* c, int32_t in_hcu, int32_t in_mcu, int32_t out_hcu,
                          int32_t out_mcu, int32_t max_batch) {
    if (!c) return;
    memset(c, 0, sizeof *c);
    c->in_hcu = in_hcu;
    c->in_mcu = in_mcu;
    c->out_hcu = out_hcu;
    c->out_mcu = out_mcu;
    c->max_batch = max_batch;
    c->alpha = 1e-3f;
    c->n_cycles = 1;
    c->gain = 1.0f;
    c->bias_gain = 1.0f;
    c->eps = 1e-8f;
    c->pi_init = 0.0f;
    c->pj_init = 0.0f;
    c->init_noise = 0.1f;
    c->seed = 0;
    c->n_swaps = 1;
    c->storage = BCPNN_STORE_F32;
}

const char* bcpnn_last_error(void) { return g_error.c_str(); }

bcpnn_status bcpnn_layer_create(const bcpnn_config* cfg, const uint8_t* mask_host,
                                void* hip_stream, bcpnn_layer** out) {
    if (!out) return fail(BCPNN_EINVAL, "out is NULL");
    *out = nullptr;
    if (const char* why = check_config(cfg)) return fail(BCPNN_EINVAL, "%s", why);
    std::vector<int32_t> list, count;
    int32_t max_active = 0;
    if (const char* why = build_active_lists(*cfg, mask_host, list, count, max_active))
        return fail(BCPNN_EINVAL, "%s", why);

    bcpnn_layer* L = new bcpnn_layer();
    L->max_active = max_active;
    L->full_mask = mask_is_full(*cfg, count);
    L->cfg = *cfg;
    L->g = Geometry{cfg->in_hcu, cfg->in_mcu, cfg->out_hcu, cfg->out_mcu,
                    (int64_t)cfg->in_hcu * cfg->in_mcu, (int64_t)cfg->out_hcu * cfg->out_mcu};
    L->stream = (hipStream_t)hip_stream;
    L->drop_bits = bcpnn::storage_drop_bits(cfg->storage);
    const Geometry& g = L->g;
    const size_t E = (size_t)g.n_in * (size_t)g.n_out;
    const size_t hh = (size_t)cfg->in_hcu * cfg->out_hcu;

    hipError_t e = hipSuccess;
    for (int k = 0; k < 2 && e == hipSuccess; ++k) {
        e = dalloc(&L->pi[k], (size_t)g.n_in);
        if (e == hipSuccess) e = dalloc(&L->pj[k], (size_t)g.n_out);
    }
    if (e == hipSuccess) e = dalloc(&L->pij, E);
    if (e == hipSuccess) e = dalloc(&L->w, E);
    if (e == hipSuccess) e = dalloc(&L->b, (size_t)g.n_out);
    if (e == hipSuccess) e = dalloc(&L->mask, hh);
    if (e == hipSuccess) e = dalloc(&L->act_list, hh);
    if (e == hipSuccess) e = dalloc(&L->act_count, (size_t)cfg->out_hcu);
    if (e == hipSuccess) e = dalloc(&L->swap_count, (size_t)cfg->out_hcu);
    if (e == hipSuccess) e = dalloc(&L->mi, hh);
    if (e == hipSuccess) e = dalloc(&L->pair_error, 1);
    if (e == hipSuccess) e = hipMemsetAsync(L->pair_error, 0, sizeof(int32_t), L->stream);
    // split operands in fragment order: 1 KiB per 32 units and 16 batch rows; the units past
    // the layer in the last block are never written and must read as zero
    const int32_t n_ks = (cfg->max_batch + 15) / 16;
    const size_t n_rt = (size_t)n_ks;
    const size_t xf = (size_t)((g.n_in + 31) / 32) * n_rt * 512;
    const size_t tf = (size_t)((g.n_out + 31) / 32) * n_rt * 512;
    for (int k = 0; k < kSets; ++k) {
        bcpnn::TraceOperands& o = L->ops[k];
        o.n_ks = n_ks;
        o.pair_error = L->pair_error;
        if (e == hipSuccess) e = dalloc(&o.x_hi, xf);
        if (e == hipSuccess) e = dalloc(&o.x_lo, xf);
        if (e == hipSuccess) e = dalloc(&o.t_hi, tf);
        if (e == hipSuccess) e = dalloc(&o.t_lo, tf);
        if (e == hipSuccess) e = dalloc(&o.x_sum, n_rt * g.n_in);
        if (e == hipSuccess) e = dalloc(&o.t_sum, n_rt * g.n_out);
        if (e == hipSuccess) e = hipMemsetAsync(o.x_hi, 0, xf * sizeof(uint16_t), L->stream);
        if (e == hipSuccess) e = hipMemsetAsync(o.x_lo, 0, xf * sizeof(uint16_t), L->stream);
        if (e == hipSuccess) e = hipMemsetAsync(o.t_hi, 0, tf * sizeof(uint16_t), L->stream);
        if (e == hipSuccess) e = hipMemsetAsync(o.t_lo, 0, tf * sizeof(uint16_t), L->stream);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&L->sweep_done[k], hipEventDisableTiming);
        L->set_sweep[k] = -1;
    }
    if (e == hipSuccess) e = hipEventCreateWithFlags(&L->sweep_ready, hipEventDisableTiming);
    // default priority; non-blocking, so that it never waits for a legacy default stream
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&L->side, hipStreamNonBlocking);
    // A small layer's sweep keeps one workgroup (one wave per SIMD) resident per CU, which
    // leaves room on every CU for the support and active-block workgroups of the batches it
    // overlaps, and still finishes within them.  A large layer's sweep is the longer stream;
    // it takes the whole machine in 128 x 128 tiles with operands staged through LDS.
    int dev = 0, n_cu = 0;
    if (e == hipSuccess) e = hipGetDevice(&dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&L->clock_khz, hipDeviceAttributeWallClockRate, dev);
    if (e == hipSuccess && L->clock_khz <= 0) e = hipErrorInvalidValue;
    const int64_t blocks = ((g.n_in + 31) / 32) * ((g.n_out + 31) / 32);
    if (e == hipSuccess) L->sweep_wgs = blocks <= kSmallSweepBlocksPerCu * (int64_t)n_cu ? n_cu : -1;
    // this device's static scratch, resolved here (the device is current) for the
    // non-allocating structural update
    if (e == hipSuccess) e = static_scratch(dev, &L->scratch);
    // complement pairs: a small layer's active-block kernel splits the rows of each pair over
    // two waves (it is bound by latency, not by its matrix work)
    const int pair_mode = !cfg->complement_pairs ? bcpnn::kUnpaired
                          : L->sweep_wgs > 0     ? bcpnn::kPairsSplit
                                                 : bcpnn::kPairs;
    for (int k = 0; k < kSets; ++k) L->ops[k].paired = pair_mode;
    if (e != hipSuccess) {
        free_layer(L);
        return fail(e == hipErrorOutOfMemory ? BCPNN_ENOMEM : BCPNN_EDEVICE,
                    "device allocation failed: %s", hipGetErrorString(e));
    }

    std::vector<uint8_t> mask(hh, 1);
    if (mask_host) memcpy(mask.data(), mask_host, hh);
    const double pi0d = cfg->pi_init > 0.0f ? (double)cfg->pi_init : 1.0 / cfg->in_mcu;
    const double pj0d = cfg->pj_init > 0.0f ? (double)cfg->pj_init : 1.0 / cfg->out_mcu;
    const float pi0 = (float)pi0d, pj0 = (float)pj0d;
    const float pij0 = (float)((double)pi0 * (double)pj0);
    std::vector<float> pi_h((size_t)g.n_in, pi0), pj_h((size_t)g.n_out, pj0);

    auto run = [&]() -> bcpnn_status {
        HIP_TRY(L, hipMemcpyAsync(L->mask, mask.data(), hh, hipMemcpyHostToDevice, L->stream));
        HIP_TRY(L, hipMemcpyAsync(L->act_list, list.data(), hh * sizeof(int32_t),
                                  hipMemcpyHostToDevice, L->stream));
        HIP_TRY(L, hipMemcpyAsync(L->act_count, count.data(), count.size() * sizeof(int32_t),
                                  hipMemcpyHostToDevice, L->stream));
        HIP_TRY(L, hipMemcpyAsync(L->pi[0], pi_h.data(), pi_h.size() * sizeof(float),
                                  hipMemcpyHostToDevice, L->stream));
        HIP_TRY(L, hipMemcpyAsync(L->pj[0], pj_h.data(), pj_h.size() * sizeof(float),
                                  hipMemcpyHostToDevice, L->stream));
        HIP_TRY(L, bcpnn::launch_init_state(L->stream, g, L->mask, pij0, cfg->init_noise, cfg->seed,
                                            L->drop_bits, L->pij, L->w));
        HIP_TRY(L, bcpnn::launch_bias(L->stream, g, L->pj[0], cfg->eps, cfg->bias_gain, L->b));
        HIP_TRY(L, hipStreamSynchronize(L->stream));
        return BCPNN_OK;
    };
    const bcpnn_status st = run();
    if (st != BCPNN_OK) {
        (void)hipStreamSynchronize(L->stream);
        free_layer(L);
        return st;
    }
    *out = L;
    return BCPNN_OK;
}

void bcpnn_layer_destroy(bcpnn_layer* L) {
    if (!L) return;
    if (!L->failed) (void)join_side(L);
    (void)hipStreamSynchronize(L->stream);
    if (L->side) (void)hipStreamSynchronize(L->side);
    free_layer(L);
}

bcpnn_status bcpnn_forward(bcpnn_layer* L, const float* x_dev, int32_t B, float* y_dev,
                           float* s_dev) {
    if (bcpnn_status st = usable(L)) return st;
    if (!x_dev || !y_dev) return fail(BCPNN_EINVAL, "x_dev and y_dev are required");
    if (misaligned(x_dev) || misaligned(y_dev) || misaligned(s_dev))
        return fail(BCPNN_EINVAL, "device buffers must be 16-byte aligned");
    if (bcpnn_status st = check_batch(L, B)) return st;
    HIP_TRY(L, bcpnn::launch_support(L->stream, L->g, x_dev, B, L->w, L->b, L->act_list,
                                     L->act_count, L->max_active, L->cfg.gain, 0, y_dev, s_dev,
                                     nullptr, nullptr, nullptr));
    return BCPNN_OK;
}

bcpnn_status bcpnn_train_batch(bcpnn_layer* L, const float* x_dev, int32_t B,
                               const float* target_dev, float* y_dev) {
    if (bcpnn_status st = usable(L)) return st;
    if (!x_dev) return fail(BCPNN_EINVAL, "x_dev is required");
    if (misaligned(x_dev) || misaligned(target_dev) || misaligned(y_dev))
        return fail(BCPNN_EINVAL, "device buffers must be 16-byte aligned");
    if (bcpnn_status st = check_batch(L, B)) return st;
    float* y = y_dev;                    // nullable: the activities then stay on the chip
    const int set = L->ops_cur;
    // the operand set is free once the sweep that read it last has run
    if (L->set_sweep[set] >= 0) HIP_TRY(L, wait_sweep(L, L->set_sweep[set]));
    L->set_sweep[set] = -1;
    unsigned long long* s_stamp = nullptr;
    HIP_TRY(L, timer_stamp(L, BCPNN_KERNEL_SUPPORT, &s_stamp));
    HIP_TRY(L, bcpnn::launch_support(L->stream, L->g, x_dev, B, L->w, L->b, L->act_list,
                                     L->act_count, L->max_active, L->cfg.gain, 0, y, nullptr,
                                     nullptr, target_dev, &L->ops[set], nullptr, nullptr,
                                     s_stamp));
    const double a_eff = 1.0 - pow(1.0 - (double)L->cfg.alpha, (double)L->cfg.n_cycles);
    bcpnn::TraceArgs a;
    a.ops = L->ops[set];
    a.B = B;
    a.a_eff = (float)a_eff;
    a.c1 = (float)(1.0 - a_eff);
    a.inv_b = (float)(1.0 / B);
    a.c2 = (float)(a_eff / B);
    a.pi_old = L->pi[L->cur];
    a.pj_old = L->pj[L->cur];
    a.pi_new = L->pi[1 - L->cur];
    a.pj_new = L->pj[1 - L->cur];
    a.pij = L->pij;
    a.w = L->w;
    a.b = L->b;
    a.mask = L->mask;
    a.eps = L->cfg.eps;
    a.bias_gain = L->cfg.bias_gain;
    a.drop_bits = L->drop_bits;
    a.stamp = nullptr;
    if (!L->full_mask) {
        // The silent elements: swept once per kMaxSweepBatches batches on the side stream,
        // which needs only the operands (written above) and touches no element the active
        // kernel below writes.
        L->pend[L->n_pend++] = bcpnn_layer::Pending{set, B, a.c1, a.c2};
        if (L->n_pend == bcpnn::kMaxSweepBatches) HIP_TRY(L, launch_pending_sweep(L));
    }
    HIP_TRY(L, timer_stamp(L, BCPNN_KERNEL_ACTIVE, &a.stamp));
    HIP_TRY(L, bcpnn::launch_trace_active(L->stream, L->g, a, L->act_list, L->act_count,
                                          L->max_active, nullptr, nullptr));
    L->cur = 1 - L->cur;
    L->ops_cur = (set + 1) % kSets;
    return BCPNN_OK;
}

bcpnn_status bcpnn_recompute_weights(bcpnn_layer* L) {
    if (bcpnn_status st = usable(L)) return st;
    HIP_TRY(L, join_side(L));
    hipEvent_t t0, t1;
    HIP_TRY(L, timer_events(L, BCPNN_KERNEL_WEIGHTS, &t0, &t1));
    HIP_TRY(L, bcpnn::launch_recompute_weights(L->stream, L->g, L->mask, L->pi[L->cur],
                                               L->pj[L->cur], L->pij, L->cfg.eps,
                                               L->cfg.bias_gain, L->drop_bits, L->w, L->b,
                                               t0, t1));
    return BCPNN_OK;
}

bcpnn_status bcpnn_structural_update(bcpnn_layer* L, int32_t* n_swapped_host) {
    if (bcpnn_status st = usable(L)) return st;
    HIP_TRY(L, join_side(L));
    // timed span: the start of the MI kernel to the end of the swap kernel (or of MI alone)
    hipEvent_t t0, t1;
    HIP_TRY(L, timer_events(L, BCPNN_KERNEL_STRUCTURAL, &t0, &t1));
    const bool swaps = L->cfg.n_swaps > 0;
    HIP_TRY(L, bcpnn::launch_mutual_information(L->stream, L->g, L->pi[L->cur], L->pj[L->cur],
                                                L->pij, L->cfg.eps, L->mi, t0));
    if (t1 && !swaps) HIP_TRY(L, hipEventRecord(t1, L->stream));
    L->mi_valid = true;
    if (swaps)
        HIP_TRY(L, bcpnn::launch_plasticity_swap(L->stream, L->g, L->mi, L->cfg.n_swaps,
                                                 L->pi[L->cur], L->pj[L->cur], L->pij,
                                                 L->cfg.eps, L->drop_bits, L->mask, L->w,
                                                 L->act_list, L->act_count, L->swap_count, t1));
    if (n_swapped_host) {
        *n_swapped_host = 0;
        std::vector<int32_t> c((size_t)L->cfg.out_hcu);
        if (swaps)
            HIP_TRY(L, hipMemcpyAsync(c.data(), L->swap_count, c.size() * sizeof(int32_t),
                                      hipMemcpyDeviceToHost, L->stream));
        HIP_TRY(L, read_input_check(L));
        HIP_TRY(L, hipStreamSynchronize(L->stream));
        if (bcpnn_status st = input_check_result(L)) return st;
        if (swaps)
            for (int32_t v : c) *n_swapped_host += v;
    }
    return BCPNN_OK;
}

bcpnn_status bcpnn_structural_update_static(bcpnn_layer* L, int32_t* n_swapped_dev) {
    if (bcpnn_status st = usable(L)) return st;
    if (((uintptr_t)n_swapped_dev & 3u) != 0)
        return fail(BCPNN_EINVAL, "n_swapped_dev must be 4-byte aligned");
    const size_t hh = (size_t)L->cfg.in_hcu * L->cfg.out_hcu;
    const size_t mi_bytes = (hh * sizeof(double) + 255) & ~(size_t)255;
    const size_t need = mi_bytes + (size_t)L->cfg.out_hcu * sizeof(int32_t);
    if (need > kStaticScratchBytes)
        return fail(BCPNN_EINVAL,
                    "structural_update_static needs %zu bytes of scratch (in_hcu * out_hcu * 8 + "
                    "out_hcu * 4, rounded) but its static scratch holds %zu; use "
                    "bcpnn_structural_update", need, kStaticScratchBytes);
    if (!L->scratch) return fail(BCPNN_EDEVICE, "static scratch not resolved on this device");
    double* mi = reinterpret_cast<double*>(L->scratch);
    int32_t* counts = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(L->scratch) + mi_bytes);
    HIP_TRY(L, join_side(L, false));
    HIP_TRY(L, bcpnn::launch_mutual_information(L->stream, L->g, L->pi[L->cur], L->pj[L->cur],
                                                L->pij, L->cfg.eps, mi));
    if (L->cfg.n_swaps > 0)
        HIP_TRY(L, bcpnn::launch_plasticity_swap(L->stream, L->g, mi, L->cfg.n_swaps,
                                                 L->pi[L->cur], L->pj[L->cur], L->pij,
                                                 L->cfg.eps, L->drop_bits, L->mask, L->w,
                                                 L->act_list, L->act_count, counts));
    if (n_swapped_dev)
        HIP_TRY(L, bcpnn::launch_count_sum(L->stream, counts,
                                           L->cfg.n_swaps > 0 ? L->cfg.out_hcu : 0,
                                           n_swapped_dev));
    L->mi_valid = false;                 // the scores stay in the shared scratch only
    return BCPNN_OK;
}

bcpnn_status bcpnn_readout(bcpnn_layer* L, const float* x_dev, int32_t B, int32_t* winner_dev) {
    if (bcpnn_status st = usable(L)) return st;
    if (!x_dev || !winner_dev) return fail(BCPNN_EINVAL, "x_dev and winner_dev are required");
    if (misaligned(x_dev) || misaligned(winner_dev))
        return fail(BCPNN_EINVAL, "device buffers must be 16-byte aligned");
    if (bcpnn_status st = check_batch(L, B)) return st;
    HIP_TRY(L, bcpnn::launch_support(L->stream, L->g, x_dev, B, L->w, L->b, L->act_list,
                                     L->act_count, L->max_active, L->cfg.gain, 1, nullptr,
                                     nullptr, winner_dev, nullptr, nullptr));
    return BCPNN_OK;
}

bcpnn_status bcpnn_flush(bcpnn_layer* L) {
    if (bcpnn_status st = usable(L)) return st;
    HIP_TRY(L, join_side(L));
    return BCPNN_OK;
}

bcpnn_status bcpnn_get_state(bcpnn_layer* L, const bcpnn_state_view* v) {
    if (bcpnn_status st = usable(L)) return st;
    if (!v) return fail(BCPNN_EINVAL, "view is NULL");
    const Geometry& g = L->g;
    const size_t E = (size_t)g.n_in * (size_t)g.n_out;
    const size_t hh = (size_t)L->cfg.in_hcu * L->cfg.out_hcu;
    auto d2h = [&](void* dst, const void* src, size_t bytes) {
        return dst ? hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, L->stream) : hipSuccess;
    };
    HIP_TRY(L, join_side(L));
    HIP_TRY(L, d2h(v->pi, L->pi[L->cur], (size_t)g.n_in * sizeof(float)));
    HIP_TRY(L, d2h(v->pj, L->pj[L->cur], (size_t)g.n_out * sizeof(float)));
    HIP_TRY(L, d2h(v->pij, L->pij, E * sizeof(float)));
    HIP_TRY(L, d2h(v->w, L->w, E * sizeof(float)));
    HIP_TRY(L, d2h(v->b, L->b, (size_t)g.n_out * sizeof(float)));
    HIP_TRY(L, d2h(v->mask, L->mask, hh));
    HIP_TRY(L, read_input_check(L));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    return input_check_result(L);
}

bcpnn_status bcpnn_set_state(bcpnn_layer* L, const bcpnn_state_view* v) {
    if (bcpnn_status st = usable(L)) return st;
    if (!v || !v->pi || !v->pj || !v->pij || !v->w || !v->b || !v->mask)
        return fail(BCPNN_EINVAL, "set_state needs all six arrays");
    std::vector<int32_t> list, count;
    int32_t max_active = 0;
    if (const char* why = build_active_lists(L->cfg, v->mask, list, count, max_active))
        return fail(BCPNN_EINVAL, "%s", why);
    const Geometry& g = L->g;
    const size_t E = (size_t)g.n_in * (size_t)g.n_out;
    const size_t hh = (size_t)L->cfg.in_hcu * L->cfg.out_hcu;
    HIP_TRY(L, join_side(L));
    HIP_TRY(L, read_input_check(L));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    if (bcpnn_status st = input_check_result(L)) return st;
    HIP_TRY(L, hipMemcpyAsync(L->pi[L->cur], v->pi, (size_t)g.n_in * sizeof(float),
                              hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->pj[L->cur], v->pj, (size_t)g.n_out * sizeof(float),
                              hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->pij, v->pij, E * sizeof(float), hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->w, v->w, E * sizeof(float), hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->b, v->b, (size_t)g.n_out * sizeof(float), hipMemcpyHostToDevice,
                              L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->mask, v->mask, hh, hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->act_list, list.data(), hh * sizeof(int32_t),
                              hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, hipMemcpyAsync(L->act_count, count.data(), count.size() * sizeof(int32_t),
                              hipMemcpyHostToDevice, L->stream));
    HIP_TRY(L, bcpnn::launch_apply_mask(L->stream, g, L->mask, L->w));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    L->max_active = max_active;
    L->full_mask = mask_is_full(L->cfg, count);
    L->mi_valid = false;
    return BCPNN_OK;
}

bcpnn_status bcpnn_get_mi(bcpnn_layer* L, double* mi_host) {
    if (bcpnn_status st = usable(L)) return st;
    if (!mi_host) return fail(BCPNN_EINVAL, "mi_host is NULL");
    if (!L->mi_valid) return fail(BCPNN_EINVAL, "no structural update since the state was set");
    const size_t hh = (size_t)L->cfg.in_hcu * L->cfg.out_hcu;
    HIP_TRY(L, hipMemcpyAsync(mi_host, L->mi, hh * sizeof(double), hipMemcpyDeviceToHost, L->stream));
    HIP_TRY(L, read_input_check(L));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    return input_check_result(L);
}

bcpnn_status bcpnn_profile_enable(bcpnn_layer* L, int32_t enable) {
    if (bcpnn_status st = usable(L)) return st;
    if (enable < 0) return fail(BCPNN_EINVAL, "profile period must be >= 0");
    L->profile_every = enable;
    for (auto& tm : L->timers) tm.launches = 0;
    return BCPNN_OK;
}

bcpnn_status bcpnn_profile_read_kernel(bcpnn_layer* L, int32_t kernel, double* total_ms,
                                       int32_t* launches) {
    if (bcpnn_status st = usable(L)) return st;
    if (!total_ms || !launches) return fail(BCPNN_EINVAL, "total_ms and launches are required");
    if (kernel < BCPNN_KERNEL_SWEEP || kernel > BCPNN_KERNEL_STRUCTURAL)
        return fail(BCPNN_EINVAL, "unknown kernel %d", kernel);
    // every launch so far complete on both streams; queued silent updates stay queued, so
    // that reading the timers leaves the schedule of the sweeps as it is
    HIP_TRY(L, read_input_check(L));
    HIP_TRY(L, hipStreamSynchronize(L->stream));
    HIP_TRY(L, hipStreamSynchronize(L->side));
    if (bcpnn_status st = input_check_result(L)) return st;
    bcpnn_layer::KernelTimer& tm = L->timers[kernel];
    double sum = 0.0;
    if (stamped(kernel))
        HIP_TRY(L, read_stamps(L, tm, &sum));
    else
        for (size_t k = 0; k < tm.used; ++k) {
            float ms = 0.0f;
            HIP_TRY(L, hipEventElapsedTime(&ms, tm.events[k].first, tm.events[k].second));
            sum += ms;
        }
    *total_ms = sum;
    *launches = (int32_t)tm.used;
    tm.used = 0;
    return BCPNN_OK;
}

bcpnn_status bcpnn_profile_read(bcpnn_layer* L, double* total_ms, int32_t* launches) {
    if (bcpnn_status st = usable(L)) return st;
    return bcpnn_profile_read_kernel(L, L->full_mask ? BCPNN_KERNEL_ACTIVE : BCPNN_KERNEL_SWEEP,
                                     total_ms, launches);
}

}  // extern "C"
