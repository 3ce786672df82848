// Capacity-constrained, bandwidth-aware placement of the experience buffer
// (Sec. 5) on one GPU host: microbenchmarks of the ingestion and delivery legs
// of each memory tier (Sec. 5.1, effective bandwidth measured on the deployment
// stack), and the linear scan of Alg. 1 over the candidate placements
// (Sec. 5.2, Eq. (placement_opt_clean)).  Host code.
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <unistd.h>

#include "common.h"

namespace conduit {

namespace {

// bytes the host can still hand out: MemAvailable of /proc/meminfo, else the
// free physical pages
double host_available_bytes() {
    if (FILE* f = std::fopen("/proc/meminfo", "r")) {
        char key[64];
        long long kib = 0;
        char unit[16];
        while (std::fscanf(f, "%63s %lld %15s", key, &kib, unit) == 3) {
            if (std::strcmp(key, "MemAvailable:") == 0) {
                std::fclose(f);
                return (double)kib * 1024.0;
            }
        }
        std::fclose(f);
    }
    const long pages = sysconf(_SC_AVPHYS_PAGES), page = sysconf(_SC_PAGESIZE);
    return pages > 0 && page > 0 ? (double)pages * (double)page : 0.0;
}

using Clock = std::chrono::steady_clock;

double seconds_since(Clock::time_point t0) { return std::chrono::duration<double>(Clock::now() - t0).count(); }

// Resources of one profile run, released by the destructor.
struct Probe {
    size_t n = 0;
    void* d0 = nullptr;   // HBM
    void* d1 = nullptr;   // HBM
    void* pin = nullptr;  // pinned host
    void* q0 = nullptr;   // pageable host
    void* q1 = nullptr;   // pageable host
    hipStream_t s = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    ~Probe() {
        if (s) (void)hipStreamSynchronize(s);
        if (d0) (void)hipFree(d0);
        if (d1) (void)hipFree(d1);
        if (pin) (void)hipHostFree(pin);
        std::free(q0);
        std::free(q1);
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
        if (s) (void)hipStreamDestroy(s);
    }
};

}  // namespace

}  // namespace conduit

using namespace conduit;

extern "C" conduit_status conduit_placement_profile(int64_t bytes, int32_t reps, conduit_place_profile* out) {
    if (!out || bytes < (1 << 20) || reps < 1) return report_error(CONDUIT_EINVAL, "need out, bytes >= 1 MiB, reps >= 1");
    Probe P;
    P.n = (size_t)bytes;
    size_t hbm_free = 0, hbm_total = 0;
    hipError_t e = hipMemGetInfo(&hbm_free, &hbm_total);
    if (e == hipSuccess) e = hipMalloc(&P.d0, P.n);
    if (e == hipSuccess) e = hipMalloc(&P.d1, P.n);
    if (e == hipSuccess) e = hipHostMalloc(&P.pin, P.n, hipHostMallocDefault);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return report_error(CONDUIT_ENOMEM, "profile buffers could not be allocated");
    }
    P.q0 = std::malloc(P.n);
    P.q1 = std::malloc(P.n);
    if (!P.q0 || !P.q1) return report_error(CONDUIT_ENOMEM, "pageable profile buffers could not be allocated");
    std::memset(P.q0, 1, P.n);  // fault the pages in before timing
    std::memset(P.q1, 2, P.n);
    std::memset(P.pin, 3, P.n);
    e = hipStreamCreateWithFlags(&P.s, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipEventCreate(&P.e0);
    if (e == hipSuccess) e = hipEventCreate(&P.e1);
    if (e == hipSuccess) e = hipMemsetAsync(P.d0, 4, P.n, P.s);
    if (e == hipSuccess) e = hipStreamSynchronize(P.s);
    if (e != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(e));
    const double nb = (double)P.n;
    // a leg the device performs, timed on the device (best of reps)
    auto dev_leg = [&](void* dst, const void* src, double* bw) {
        hipError_t r = hipMemcpyAsync(dst, src, P.n, hipMemcpyDefault, P.s);  // warm-up
        float best = 0.0f;
        for (int i = 0; i < reps && r == hipSuccess; ++i) {
            float ms = 0.0f;
            r = hipEventRecord(P.e0, P.s);
            if (r == hipSuccess) r = hipMemcpyAsync(dst, src, P.n, hipMemcpyDefault, P.s);
            if (r == hipSuccess) r = hipEventRecord(P.e1, P.s);
            if (r == hipSuccess) r = hipEventSynchronize(P.e1);
            if (r == hipSuccess) r = hipEventElapsedTime(&ms, P.e0, P.e1);
            if (r == hipSuccess && (i == 0 || ms < best)) best = ms;
        }
        *bw = r == hipSuccess && best > 0.0f ? nb / ((double)best * 1e-3) : 0.0;
        return r;
    };
    // a leg that involves pageable memory: the runtime stages it through its
    // own pinned buffers on the host's time, so it is timed by the host clock
    // around a synchronous copy
    auto staged_leg = [&](void* dst, const void* src, double* bw) {
        hipError_t r = hipMemcpy(dst, src, P.n, hipMemcpyDefault);
        double best = 0.0;
        for (int i = 0; i < reps && r == hipSuccess; ++i) {
            const Clock::time_point t0 = Clock::now();
            r = hipMemcpy(dst, src, P.n, hipMemcpyDefault);
            const double t = seconds_since(t0);
            if (r == hipSuccess && (i == 0 || t < best)) best = t;
        }
        *bw = r == hipSuccess && best > 0.0 ? nb / best : 0.0;
        return r;
    };
    // a leg the CPU performs (a CPU actor writing into a host tier)
    auto host_leg = [&](void* dst, const void* src, double* bw) {
        std::memcpy(dst, src, P.n);
        double best = 0.0;
        for (int i = 0; i < reps; ++i) {
            const Clock::time_point t0 = Clock::now();
            std::memcpy(dst, src, P.n);
            const double t = seconds_since(t0);
            if (i == 0 || t < best) best = t;
        }
        *bw = best > 0.0 ? nb / best : 0.0;
    };
    conduit_place_profile r{};
    constexpr int HBM = CONDUIT_PLACE_HBM, PIN = CONDUIT_PLACE_HOST_PINNED, PAGE = CONDUIT_PLACE_HOST_PAGEABLE;
    // GPU actor (rollouts in HBM) -> buffer
    e = dev_leg(P.d1, P.d0, &r.bw_in[1][HBM]);
    if (e == hipSuccess) e = dev_leg(P.pin, P.d0, &r.bw_in[1][PIN]);
    if (e == hipSuccess) e = staged_leg(P.q1, P.d0, &r.bw_in[1][PAGE]);
    // CPU actor (rollouts in pageable memory) -> buffer
    if (e == hipSuccess) e = staged_leg(P.d1, P.q0, &r.bw_in[0][HBM]);
    host_leg(P.pin, P.q0, &r.bw_in[0][PIN]);
    host_leg(P.q1, P.q0, &r.bw_in[0][PAGE]);
    // buffer -> learner GPU
    r.bw_out[HBM] = r.bw_in[1][HBM];
    if (e == hipSuccess) e = dev_leg(P.d1, P.pin, &r.bw_out[PIN]);
    r.bw_out[PAGE] = r.bw_in[0][HBM];
    if (e != hipSuccess) return report_error(CONDUIT_EDEVICE, hipGetErrorString(e));
    r.mem[HBM] = (double)hbm_free;
    r.mem[PIN] = r.mem[PAGE] = host_available_bytes();
    *out = r;
    return CONDUIT_OK;
}

extern "C" conduit_status conduit_place(const conduit_place_profile* prof, int32_t actor_on_gpu, int64_t capacity,
                                        double sample_bytes, const int32_t* candidates, int32_t n, int32_t* choice,
                                        double* t_transfer) {
    if (!prof || !candidates || !choice || n < 1) return report_error(CONDUIT_EINVAL, "NULL argument or no candidates");
    if (actor_on_gpu != 0 && actor_on_gpu != 1) return report_error(CONDUIT_EINVAL, "actor_on_gpu must be 0 or 1");
    if (capacity < 0 || !(sample_bytes > 0.0) || !std::isfinite(sample_bytes))
        return report_error(CONDUIT_EINVAL, "capacity must be >= 0 and sample_bytes > 0");
    for (int i = 0; i < n; ++i) {
        const int p = candidates[i];
        if (p < 0 || p >= CONDUIT_PLACEMENTS) return report_error(CONDUIT_EINVAL, "unknown placement");
        if (!(prof->bw_in[actor_on_gpu][p] > 0.0) || !(prof->bw_out[p] > 0.0))
            return report_error(CONDUIT_EINVAL, "bandwidths of a scanned placement must be > 0");
    }
    // Alg. 1: keep the first feasible candidate of least transfer latency
    const double need = (double)capacity * sample_bytes;
    int best = -1;
    double t_min = INFINITY;
    for (int i = 0; i < n; ++i) {
        const int p = candidates[i];
        const double t = sample_bytes / prof->bw_in[actor_on_gpu][p] + sample_bytes / prof->bw_out[p];
        if (t_transfer) t_transfer[i] = t;
        if (need <= prof->mem[p] && t < t_min) {
            t_min = t;
            best = p;
        }
    }
    *choice = best;
    return CONDUIT_OK;
}
