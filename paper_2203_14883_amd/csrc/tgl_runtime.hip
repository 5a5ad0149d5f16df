// tgl_runtime.hip -- version, status strings, kernel timers and the
// single-block scan of tile partials.
#include <mutex>
#include <vector>

#include "tgl_internal.hpp"

namespace tgl {

// ---- scan of tile partials: one block of 1024 threads ----
__global__ __launch_bounds__(1024) void scan_partials_kernel(int64_t *__restrict__ partials,
                                                             int64_t nb,
                                                             int64_t *__restrict__ total_out) {
    __shared__ int64_t lds[1024 / kWave];
    const int64_t per = (nb + 1023) / 1024;
    const int64_t b0 = static_cast<int64_t>(threadIdx.x) * per;
    const int64_t b1 = b0 + per < nb ? b0 + per : nb;
    int64_t sum = 0;
    for (int64_t i = b0; i < b1; i++) sum += partials[i];
    // block-wide exclusive scan of the per-thread sums
    const int64_t inc = wave_inclusive_sum(sum);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) lds[w] = inc;
    __syncthreads();
    int64_t before = 0, all = 0;
    for (int i = 0; i < 1024 / kWave; i++) {
        const int64_t x = lds[i];
        if (i < w) before += x;
        all += x;
    }
    int64_t run = before + inc - sum;
    for (int64_t i = b0; i < b1; i++) {
        const int64_t x = partials[i];
        partials[i] = run;
        run += x;
    }
    if (threadIdx.x == 0 && total_out) *total_out = all;
}

void launch_scan_partials(int64_t *partials, int64_t nb, int64_t *total_out, hipStream_t s) {
    scan_partials_kernel<<<1, 1024, 0, s>>>(partials, nb, total_out);
}

// ---- kernel timers ----
namespace {
struct TimerState {
    std::mutex mu;
    bool on = false;
    std::vector<hipEvent_t> ev;        // 2 per slot
    std::vector<int> kind;             // kind of each used slot
    int used = 0;
    uint32_t kinds = ~0u;              // bit k set: launches of kind k are recorded
};
TimerState &timers() {
    static TimerState t;
    return t;
}
}  // namespace

int timer_begin(int k, hipStream_t s) {
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    if (!t.on || !((t.kinds >> k) & 1u) || t.used * 2 + 1 >= static_cast<int>(t.ev.size())) return -1;
    const int slot = t.used++;
    t.kind[slot] = k;
    if (hipEventRecord(t.ev[2 * slot], s) != hipSuccess) {
        t.kind[slot] = -1;
        return -1;
    }
    return slot;
}

void timer_end(int slot, hipStream_t s) {
    if (slot < 0) return;
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    if (!t.on || slot >= t.used) return;
    if (hipEventRecord(t.ev[2 * slot + 1], s) != hipSuccess) t.kind[slot] = -1;
}

}  // namespace tgl

using namespace tgl;

extern "C" {

int32_t tgl_version(void) { return 10000; }

const char *tgl_status_str(tgl_status s) {
    switch (s) {
        case TGL_OK: return "ok";
        case TGL_EINVAL: return "invalid argument";
        case TGL_ERANGE: return "build input out of range (endpoint or NaN timestamp)";
        case TGL_ENOSPACE: return "workspace too small";
        case TGL_EDEVICE: return "device error";
        default: return "unknown status";
    }
}

tgl_status tgl_timer_enable(int32_t capacity) {
    if (capacity < 1 || capacity > (1 << 20)) return TGL_EINVAL;
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    for (hipEvent_t e : t.ev) (void)hipEventDestroy(e);
    t.ev.assign(2 * static_cast<size_t>(capacity), nullptr);
    t.kind.assign(static_cast<size_t>(capacity), -1);
    for (auto &e : t.ev) {
        if (hipEventCreate(&e) != hipSuccess) {
            t.ev.clear();
            t.on = false;
            return TGL_EDEVICE;
        }
    }
    t.used = 0;
    t.kinds = ~0u;
    t.on = true;
    return TGL_OK;
}

tgl_status tgl_timer_disable(void) {
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    for (hipEvent_t e : t.ev) (void)hipEventDestroy(e);
    t.ev.clear();
    t.kind.clear();
    t.used = 0;
    t.on = false;
    return TGL_OK;
}

tgl_status tgl_timer_select(uint32_t kinds) {
    if (kinds >> TGL_TIMER_KINDS) return TGL_EINVAL;
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    t.kinds = kinds;
    return TGL_OK;
}

tgl_status tgl_timer_reset(void) {
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    t.used = 0;
    for (auto &k : t.kind) k = -1;
    return TGL_OK;
}

tgl_status tgl_timer_read(int32_t kind, double *total_ms, int64_t *launches) {
    if (kind < 0 || kind >= TGL_TIMER_KINDS || !total_ms || !launches) return TGL_EINVAL;
    TimerState &t = timers();
    std::lock_guard<std::mutex> g(t.mu);
    double sum = 0.0;
    int64_t n = 0;
    for (int i = 0; i < t.used; i++) {
        if (t.kind[i] != kind) continue;
        if (hipEventSynchronize(t.ev[2 * i + 1]) != hipSuccess) return TGL_EDEVICE;
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]) != hipSuccess) return TGL_EDEVICE;
        sum += ms;
        n++;
    }
    *total_ms = sum;
    *launches = n;
    return TGL_OK;
}

}  // extern "C"
