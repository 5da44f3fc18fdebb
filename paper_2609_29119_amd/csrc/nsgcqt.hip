// C ABI of the packed constant-Q transform: plan creation (host tables built in
// fp64, uploaded once as fp32), and the enqueue-only compute calls.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <tuple>
#include <type_traits>
#include <utility>
#include <vector>

#include "../../include/nsgcqt.h"
#include "kernels.hpp"
#include "plan.hpp"

using namespace nsg;

namespace {

thread_local std::string g_err;

int set_err(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define HIP_TRY(expr)                                                                  \
    do {                                                                               \
        hipError_t e_ = (expr);                                                        \
        if (e_ != hipSuccess)                                                          \
            return set_err(NSGCQT_EDEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Launches kernel k with the arguments converted to its parameter types and
// returns the status of this launch alone. (hipGetLastError after a launch
// would also report an error that an earlier, unrelated HIP call of the
// caller left on the thread.)
template <typename... P, typename... A>
hipError_t launch_kernel(void (*k)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t s, A&&... a) {
    static_assert(sizeof...(P) == sizeof...(A), "kernel argument count");
    std::tuple<std::decay_t<P>...> vals(std::forward<A>(a)...);
    return std::apply(
        [&](auto&... v) {
            void* args[] = {static_cast<void*>(&v)...};
            return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, args, lds, s);
        },
        vals);
}

#define LAUNCH_TRY(...)                                                                \
    do {                                                                               \
        hipError_t e_ = launch_kernel(__VA_ARGS__);                                    \
        if (e_ != hipSuccess)                                                          \
            return set_err(NSGCQT_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(e_)); \
    } while (0)

int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

}  // namespace

// Workspace of the allocation-free analysis (nsgcqt_analyse_noalloc). Host
// code never uses this name as an address: each device's copy is reached
// through the pointer that hipGetSymbolAddress returns on that device.
static __device__ __align__(256) char scratch[NSGCQT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up once per
// device (with that device current) and kept.
int scratch_address(void** out) {
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return set_err(NSGCQT_EDEVICE, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return set_err(NSGCQT_EDEVICE, std::string("hipGetSymbolAddress of the scratch array: ") +
                                               hipGetErrorString(e));
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return NSGCQT_OK;
}

}  // namespace

struct nsgcqt_plan_s {
    HostPlan h;
    bool device = false;
    int dev = -1;   // the device that holds the tables (current at creation)
    void* dmem = nullptr;
    int64_t dbytes = 0;
    Tables T{};
    const float* wA = nullptr;
    const float* wS = nullptr;
    const float* wT = nullptr;
    const float* wSa = nullptr;
    const float4* rA = nullptr;    // router factors of T and S^dagger
    const float4* rSa = nullptr;
    std::vector<hipEvent_t> events;
    int ev_next = 0;
    std::map<const void*, int> resident;   // persistent kernels: workgroups resident at once
    // independent launches of one call (band tiers, the huge-band chain) run
    // concurrently on the caller's stream and these side streams (default
    // priority), forked from and joined back into the caller's stream
    static constexpr int kSide = 3;
    hipStream_t side[kSide] = {};
    hipEvent_t fork_ev = nullptr;
    hipEvent_t join_ev[kSide] = {};
    // only for plans whose band launches are all small and whose band phase
    // is long (see schedule)
    bool fan = false;
    // launch units: the buckets, then the huge-band chain (when there are huge bands)
    std::vector<int> lane;    // stream of each unit: 0 = caller's
    std::vector<int> order;   // enqueue order of the units
    // the enqueue state above (events, the resident-block cache, the fork and
    // join events) is used by one call at a time
    std::mutex mu;
};

namespace {

// ------------------------------------------------------------------ upload
int upload(nsgcqt_plan_s* p) {
    HostPlan& h = p->h;
    struct Chunk { const void* src; int64_t bytes; int64_t off; };
    std::vector<Chunk> ch;
    int64_t total = 0;
    // guard: bytes after the table that the band kernels' fast load phases
    // may read (and ignore)
    auto add = [&](const void* src, int64_t bytes, int64_t guard = 0) {
        ch.push_back({src, bytes, total});
        total += align256((bytes > 0 ? bytes : 1) + guard);
        return ch.size() - 1;
    };
    const int64_t g1 = kFastGuard * static_cast<int64_t>(sizeof(float)), g4 = 4 * g1;
    const size_t iBands = add(h.banddev.data(), h.banddev.size() * sizeof(BandDev));
    const size_t iFfts = add(h.ffts.data(), h.ffts.size() * sizeof(FftDesc));
    const size_t iTw = add(h.twpool.data(), h.twpool.size() * sizeof(float));
    const size_t iOm = add(h.omega.data(), h.omega.size() * sizeof(float));
    const size_t iOwn = add(h.owner.data(), h.owner.size() * sizeof(int32_t));
    const size_t iBase = add(h.bandbase.data(), h.bandbase.size() * sizeof(int32_t));
    const size_t iGather = add(h.gather.data(), h.gather.size() * sizeof(int32_t));
    const size_t iCh = add(h.chirp.data(), h.chirp.size() * sizeof(float), 2 * g1);
    const size_t iK = add(h.kern.data(), h.kern.size() * sizeof(float));
    const size_t iHi = add(h.tw4_hi.data(), h.tw4_hi.size() * sizeof(float));
    const size_t iLo = add(h.tw4_lo.data(), h.tw4_lo.size() * sizeof(float));
    const size_t iWin = add(h.slicewin.data(), h.slicewin.size() * sizeof(float));
    const size_t iItems = add(h.items.data(), h.items.size() * sizeof(WorkItem));
    const size_t iBigs = add(h.bigs.data(), h.bigs.size() * sizeof(BigDesc));
    const size_t iBigItems = add(h.bigitems.data(), h.bigitems.size() * sizeof(BigItem));
    const size_t iWA = add(h.wA.data(), h.wA.size() * sizeof(float), g1);
    const size_t iWS = add(h.wS.data(), h.wS.size() * sizeof(float), g1);
    const size_t iWT = add(h.wT.data(), h.wT.size() * sizeof(float), g1);
    const size_t iWSa = add(h.wSa.data(), h.wSa.size() * sizeof(float), g1);
    const size_t iRA = add(h.rA.data(), h.rA.size() * sizeof(float), g4);
    const size_t iRSa = add(h.rSa.data(), h.rSa.size() * sizeof(float), g4);

    HIP_TRY(hipGetDevice(&p->dev));
    char* d = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&d), total);
    if (e != hipSuccess) return set_err(NSGCQT_ENOMEM, std::string("hipMalloc of plan tables: ") + hipGetErrorString(e));
    p->dmem = d;
    p->dbytes = total;
    for (const auto& c : ch)
        if (c.bytes > 0) HIP_TRY(hipMemcpy(d + c.off, c.src, c.bytes, hipMemcpyHostToDevice));
    auto at = [&](size_t i) { return static_cast<const void*>(d + ch[i].off); };
    Tables& T = p->T;
    T.bands = static_cast<const BandDev*>(at(iBands));
    T.ffts = static_cast<const FftDesc*>(at(iFfts));
    T.tw = static_cast<const float2*>(at(iTw));
    T.omega = static_cast<const float2*>(at(iOm));
    T.owner = static_cast<const int32_t*>(at(iOwn));
    T.bandbase = static_cast<const int32_t*>(at(iBase));
    T.gather = static_cast<const int4*>(at(iGather));
    T.chirp = static_cast<const float2*>(at(iCh));
    T.kern = static_cast<const float2*>(at(iK));
    T.tw4_hi = static_cast<const float2*>(at(iHi));
    T.tw4_lo = static_cast<const float2*>(at(iLo));
    T.slicewin = static_cast<const float*>(at(iWin));
    T.items = static_cast<const WorkItem*>(at(iItems));
    T.bigs = static_cast<const BigDesc*>(at(iBigs));
    T.bigitems = static_cast<const BigItem*>(at(iBigItems));
    p->wA = static_cast<const float*>(at(iWA));
    p->wS = static_cast<const float*>(at(iWS));
    p->wT = static_cast<const float*>(at(iWT));
    p->wSa = static_cast<const float*>(at(iWSa));
    p->rA = static_cast<const float4*>(at(iRA));
    p->rSa = static_cast<const float4*>(at(iRSa));
    // the fork and join events order work within this device only
    const unsigned evf = hipEventDisableTiming | hipEventDisableSystemFence;
    for (int i = 0; i < nsgcqt_plan_s::kSide; ++i) {
        HIP_TRY(hipStreamCreateWithFlags(&p->side[i], hipStreamNonBlocking));
        HIP_TRY(hipEventCreateWithFlags(&p->join_ev[i], evf));
    }
    HIP_TRY(hipEventCreateWithFlags(&p->fork_ev, evf));
    p->device = true;
    return NSGCQT_OK;
}

// Launch schedule of the band phase, from the host plan alone. Overlap pays
// when no band launch fills the GPU by itself and the band phase is long
// against the fork and join (~25 us each way): at least 6M element slots of
// band work. Then units are enqueued longest first, each onto the least
// loaded of the four streams; otherwise in bucket order on the caller's.
void schedule(nsgcqt_plan_s* p) {
    const HostPlan& h = p->h;
    std::vector<double> cost;
    int most = 0;
    for (const auto& bk : h.buckets) {
        most = std::max(most, bk.nitems);
        cost.push_back(static_cast<double>(bk.nitems) * bk.nt * bk.ept);
    }
    if (!h.bigs.empty()) cost.push_back(4.0 * static_cast<double>(h.Hn) * static_cast<double>(h.batch));
    double work = 0.0;
    for (double c : cost) work += c;
    p->fan = most < 2048 && work >= 6e6;
    p->order.resize(cost.size());
    for (size_t i = 0; i < cost.size(); ++i) p->order[i] = static_cast<int>(i);
    p->lane.assign(cost.size(), 0);
    if (!p->fan) return;
    std::stable_sort(p->order.begin(), p->order.end(), [&](int a, int b) { return cost[a] > cost[b]; });
    double load[nsgcqt_plan_s::kSide + 1] = {};
    for (int u : p->order) {
        int best = 0;
        for (int k = 1; k <= nsgcqt_plan_s::kSide; ++k)
            if (load[k] < load[best]) best = k;
        p->lane[u] = best;
        load[best] += cost[u];
    }
}

// Releases the plan's device tables, side streams and events.
int release(nsgcqt_plan_s* p) {
    hipError_t e = hipSuccess;
    auto keep = [&](hipError_t r) { if (e == hipSuccess) e = r; };
    for (int i = 0; i < nsgcqt_plan_s::kSide; ++i) {
        if (p->side[i]) keep(hipStreamDestroy(p->side[i]));
        if (p->join_ev[i]) keep(hipEventDestroy(p->join_ev[i]));
        p->side[i] = nullptr;
        p->join_ev[i] = nullptr;
    }
    if (p->fork_ev) keep(hipEventDestroy(p->fork_ev));
    p->fork_ev = nullptr;
    if (p->dmem) keep(hipFree(p->dmem));
    p->dmem = nullptr;
    if (e != hipSuccess) return set_err(NSGCQT_EDEVICE, std::string("release: ") + hipGetErrorString(e));
    return NSGCQT_OK;
}

// Spreads independent launches over the caller's stream s and the plan's
// side streams: unit u runs on s when its lane is 0, else on side stream
// lane - 1, which first waits for the work already on s; join() makes s
// wait for every side stream used.
struct Fanout {
    nsgcqt_plan_s* p;
    hipStream_t s;
    bool forked = false;
    bool used[nsgcqt_plan_s::kSide] = {};
    // the fork point precedes every launch of the phase, including those
    // that go on s itself
    int begin() {
        if (!p->fan) return NSGCQT_OK;
        HIP_TRY(hipEventRecord(p->fork_ev, s));
        forked = true;
        return NSGCQT_OK;
    }
    int stream(int u, hipStream_t* out) {
        const int k = p->fan ? p->lane[u] : 0;
        if (k == 0 || !forked) {
            *out = s;
            return NSGCQT_OK;
        }
        if (!used[k - 1]) {
            HIP_TRY(hipStreamWaitEvent(p->side[k - 1], p->fork_ev, 0));
            used[k - 1] = true;
        }
        *out = p->side[k - 1];
        return NSGCQT_OK;
    }
    int join() {
        for (int i = 0; i < nsgcqt_plan_s::kSide; ++i)
            if (used[i]) {
                HIP_TRY(hipEventRecord(p->join_ev[i], p->side[i]));
                HIP_TRY(hipStreamWaitEvent(s, p->join_ev[i], 0));
            }
        return NSGCQT_OK;
    }
};

// ---------------------------------------------------------------- launches
// Kernels with more than 64 KB of dynamic LDS get the attribute that allows
// it, once per kernel and device at the largest size asked for so far.
template <typename K>
int launch_prep(K kernel, int lds_bytes) {
    if (lds_bytes <= 64 * 1024) return NSGCQT_OK;
    static std::mutex mu;
    static std::map<std::pair<const void*, int>, int> done;
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    const auto key = std::make_pair(reinterpret_cast<const void*>(kernel), dev);
    std::lock_guard<std::mutex> lock(mu);
    auto it = done.find(key);
    if (it != done.end() && it->second >= lds_bytes) return NSGCQT_OK;
    HIP_TRY(hipFuncSetAttribute(key.first, hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes));
    done[key] = lds_bytes;
    return NSGCQT_OK;
}

// Stage timing: with events installed, kernel launch i is bracketed by
// events[2i] and events[2i + 1] on its stream; NULL entries are skipped.
void ev_start(nsgcqt_plan_s* p, hipStream_t s) {
    if (p->ev_next + 1 < static_cast<int>(p->events.size()) && p->events[p->ev_next])
        hipEventRecord(p->events[p->ev_next], s);
}
void ev_end(nsgcqt_plan_s* p, hipStream_t s) {
    if (p->ev_next + 1 < static_cast<int>(p->events.size())) {
        if (p->events[p->ev_next + 1]) hipEventRecord(p->events[p->ev_next + 1], s);
        p->ev_next += 2;
    }
}

Pass pass_a(const HostPlan& h) {
    Pass q{};
    q.L1 = static_cast<int>(h.fs4.L1); q.L2 = static_cast<int>(h.fs4.L2);
    q.lgnb = h.fs4.tile_a;
    q.ntile = static_cast<int>((h.fs4.L2 + (int64_t(1) << q.lgnb) - 1) >> q.lgnb);
    q.fft = h.fs4.fft1;
    q.ntw = h.ffts[q.fft].ntw;
    q.split = static_cast<int>(h.fs4.split);
    q.nhi4 = static_cast<int>(h.tw4_hi.size() / 2);
    q.L = static_cast<int>(h.L);
    return q;
}

Pass pass_b(const HostPlan& h) {
    Pass q = pass_a(h);
    q.lgnb = h.fs4.tile_b;
    q.ntile = static_cast<int>((h.fs4.L1 + (int64_t(1) << q.lgnb) - 1) >> q.lgnb);
    q.fft = h.fs4.fft2;
    q.ntw = h.ffts[q.fft].ntw;
    return q;
}

int lds_pass_a(const Pass& q) {
    return (q.nhi4 + (1 << q.split) + lds_slots(q.L1, q.lgnb)) * static_cast<int>(sizeof(float2));
}
int lds_pass_b(const Pass& q) {
    return (q.ntw + lds_slots(q.L2, q.lgnb)) * static_cast<int>(sizeof(float2));
}

// Workgroups of a persistent kernel that are resident on the device at once
// (cached per plan and kernel); 0 if the runtime cannot say.
template <typename K>
int resident_blocks(nsgcqt_plan_s* p, K kernel, int nt, int lds) {
    const void* key = reinterpret_cast<const void*>(kernel);
    auto it = p->resident.find(key);
    if (it != p->resident.end()) return it->second;
    int dev = 0, cus = 0, per = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, key, nt, lds) != hipSuccess)
        return 0;
    p->resident[key] = cus * per;
    return cus * per;
}

#define DISPATCH_NT(nt, KERNEL, ...)                                                         \
    switch (nt) {                                                                            \
        case 256: { auto k_ = KERNEL<256, 8 __VA_ARGS__>; if (int r_ = launch(k_)) return r_; break; } \
        case 512: { auto k_ = KERNEL<512, 8 __VA_ARGS__>; if (int r_ = launch(k_)) return r_; break; } \
        default: { auto k_ = KERNEL<1024, 8 __VA_ARGS__>; if (int r_ = launch(k_)) return r_; break; } \
    }

int run_fwd_a(nsgcqt_plan_s* p, const float* x, float2* Y, int batch, SliceIn sl, long long sig_stride,
              hipStream_t s) {
    const Pass q = pass_a(p->h);
    const int lds = lds_pass_a(q) + q.ntw * static_cast<int>(sizeof(float2));   // + stage twiddles
    auto launch = [&](auto k) -> int {
        if (int r = launch_prep(k, lds)) return r;
        const int tiles = q.ntile * batch;
        const int res = resident_blocks(p, k, p->h.fs4.nt_a, lds);
        const int grid = res > 0 ? std::min(tiles, res) : tiles;
        ev_start(p, s);
        LAUNCH_TRY(k, dim3(grid), dim3(p->h.fs4.nt_a), lds, s, x, Y, q, p->T, sl, batch, sig_stride);
        ev_end(p, s);
        return NSGCQT_OK;
    };
    if (sl.enabled) {
        // the plan keeps sliced column passes at 512 threads or fewer
        if (p->h.fs4.nt_a == 256) {
            if (int r = launch(k_fwd_a<256, 8, true>)) return r;
        } else if (p->h.fs4.nt_a == 512) {
            if (int r = launch(k_fwd_a<512, 8, true>)) return r;
        } else {
            return set_err(NSGCQT_EUNSUPPORTED, "sliced column pass above 512 threads");
        }
    } else {
        DISPATCH_NT(p->h.fs4.nt_a, k_fwd_a, , false)
    }
    return NSGCQT_OK;
}

int run_inv_a(nsgcqt_plan_s* p, const float2* W, float2* Y, int batch, hipStream_t s) {
    Pass q = pass_a(p->h);
    // tiles of 2^(lgnb-1) primary columns in [0, L2/2] and their mirrors
    if (q.lgnb >= 1) {
        const int H = 1 << (q.lgnb - 1);
        q.ntile = (q.L2 / 2 + 1 + H - 1) / H;
    } else {
        q.ntile = q.L2;
    }
    const int lds = lds_pass_a(q);
    auto launch = [&](auto k) -> int {
        if (int r = launch_prep(k, lds)) return r;
        ev_start(p, s);
        LAUNCH_TRY(k, dim3(q.ntile * batch), dim3(p->h.fs4.nt_a), lds, s, W, Y, q, p->T, batch,
                   static_cast<long long>(p->h.C));
        ev_end(p, s);
        return NSGCQT_OK;
    };
    if (p->h.gather_wide) {
        DISPATCH_NT(p->h.fs4.nt_a, k_inv_a, , true)
    } else {
        DISPATCH_NT(p->h.fs4.nt_a, k_inv_a, , false)
    }
    return NSGCQT_OK;
}

template <bool INV>
int run_pass_b(nsgcqt_plan_s* p, const float2* Y, float2* out, int batch, long long out_stride, hipStream_t s) {
    const Pass q = pass_b(p->h);
    const int lds = lds_pass_b(q);
    const float inv_L = static_cast<float>(1.0 / static_cast<double>(p->h.L));
    auto launch = [&](auto k) -> int {
        if (int r = launch_prep(k, lds)) return r;
        const int tiles = q.ntile * batch;
        const int res = resident_blocks(p, k, p->h.fs4.nt_b, lds);
        const int grid = res > 0 ? std::min(tiles, res) : tiles;
        ev_start(p, s);
        LAUNCH_TRY(k, dim3(grid), dim3(p->h.fs4.nt_b), lds, s, Y, out, q, p->T, batch,
                   out_stride, inv_L);
        ev_end(p, s);
        return NSGCQT_OK;
    };
    DISPATCH_NT(p->h.fs4.nt_b, k_pass_b, , INV)
    return NSGCQT_OK;
}

// One band tier (bucket bi) as one launch, on the stream of fan-out unit bi.
// Analysis reads the router factors rt, synthesis the weights wt.
int run_bucket(nsgcqt_plan_s* p, size_t bi, bool analysis, const float2* in, float2* out, const float4* rt,
               const float* wt, int batch, Fanout& fan) {
    const HostPlan& h = p->h;
    const Bucket& bk = h.buckets[bi];
    hipStream_t s;
    if (int r = fan.stream(static_cast<int>(bi), &s)) return r;
    const int lds = bk.lds_elems * static_cast<int>(sizeof(float2));
    const dim3 grid(bk.nitems), block(bk.nt);
    auto go = [&](auto ka, auto ks) -> int {
        ev_start(p, s);
        if (analysis) {
            if (int r = launch_prep(ka, lds)) return r;
            LAUNCH_TRY(ka, grid, block, lds, s, in, out, rt, p->T, bk.item_off, bk.nitems, batch,
                       static_cast<int>(h.L), static_cast<long long>(h.C));
        } else {
            if (int r = launch_prep(ks, lds)) return r;
            LAUNCH_TRY(ks, grid, block, lds, s, in, out, wt, p->T, bk.item_off, bk.nitems, batch,
                       static_cast<long long>(h.C));
        }
        ev_end(p, s);
        return NSGCQT_OK;
    };
    if (bk.nt == 64) return go(k_band_analysis<64, 8>, k_band_synthesis<64, 8>);
    if (bk.nt == 256 && bk.ept == 8) return go(k_band_analysis<256, 8>, k_band_synthesis<256, 8>);
    if (bk.nt == 256) return go(k_band_analysis<256, 16>, k_band_synthesis<256, 16>);
    if (bk.nt == 512) return go(k_band_analysis<512, 16>, k_band_synthesis<512, 16>);
    return go(k_band_analysis<1024, 16>, k_band_synthesis<1024, 16>);
}

// Huge bands: column pass and row pass over every huge band, then for the
// Bluestein ones the second FFT (column pass reading H2, row pass finishing).
int run_big(nsgcqt_plan_s* p, BigArgs a, int batch, hipStream_t s) {
    const HostPlan& h = p->h;
    if (h.bigs.empty()) return NSGCQT_OK;
    auto ka = k_big_a<512, 8>;
    auto kb = k_big_b<512, 8>;
    if (int r = launch_prep(ka, h.big_lds_a)) return r;
    if (int r = launch_prep(kb, h.big_lds_b)) return r;
    const int in0 = a.analysis ? kBigInRoute : kBigInCoef;
    for (int pass = 0; pass < 4; ++pass) {
        const int n = h.big_n[pass];
        if (n == 0) continue;
        ev_start(p, s);
        if (pass % 2 == 0)
            LAUNCH_TRY(ka, dim3(n), dim3(512), h.big_lds_a, s, a, p->T, h.big_off[pass], n, batch,
                       pass == 0 ? in0 : kBigInBlu2);
        else
            LAUNCH_TRY(kb, dim3(n), dim3(512), h.big_lds_b, s, a, p->T, h.big_off[pass], n, batch,
                       pass == 3 ? 1 : 0);
        ev_end(p, s);
    }
    return NSGCQT_OK;
}

BigArgs big_args(nsgcqt_plan_s* p, char* ws, int64_t hoff, int batch, bool analysis) {
    const HostPlan& h = p->h;
    BigArgs a{};
    a.H1 = reinterpret_cast<float2*>(ws + hoff);
    a.H2 = reinterpret_cast<float2*>(ws + hoff + align256(8 * h.Hn * batch));
    a.L = static_cast<int>(h.L);
    a.C = h.C;
    a.Hn = h.Hn;
    a.analysis = analysis ? 1 : 0;
    return a;
}

// The band phase of one call: every bucket and the huge-band chain, in the
// plan's schedule order and on its streams; returns with s after all of them.
int run_band_phase(nsgcqt_plan_s* p, bool analysis, const float2* in, float2* out, const float4* rt,
                   const float* wt, BigArgs a, int batch, hipStream_t s) {
    const HostPlan& h = p->h;
    Fanout fan{p, s};
    if (int r = fan.begin()) return r;
    for (int u : p->order) {
        if (u < static_cast<int>(h.buckets.size())) {
            if (int r = run_bucket(p, static_cast<size_t>(u), analysis, in, out, rt, wt, batch, fan)) return r;
        } else {
            hipStream_t sb;
            if (int r = fan.stream(u, &sb)) return r;
            if (int r = run_big(p, a, batch, sb)) return r;
        }
    }
    return fan.join();
}

// Analysis chain (T, or S^dagger with its weights) for `batch` signals or slices.
int chain_analyse(nsgcqt_plan_s* p, const float* x, float2* coeffs, const float4* rt, int batch, SliceIn sl,
                  char* ws, hipStream_t s) {
    const HostPlan& h = p->h;
    float2* Y = reinterpret_cast<float2*>(ws);
    float2* Z = reinterpret_cast<float2*>(ws + align256(8 * h.L * batch));
    if (int r = run_fwd_a(p, x, Y, batch, sl, static_cast<long long>(h.N), s)) return r;
    if (int r = run_pass_b<false>(p, Y, Z, batch, static_cast<long long>(h.L), s)) return r;
    BigArgs a = big_args(p, ws, h.off_h_an, h.spc ? h.spc : batch, true);
    a.Z = Z;
    a.cout = coeffs;
    a.rt = rt;
    if (int r = run_band_phase(p, true, Z, coeffs, rt, nullptr, a, batch, s)) return r;
    return NSGCQT_OK;
}

// Synthesis chain (S, or T^dagger with its weights); output is [batch][N] f32.
int chain_synthesise(nsgcqt_plan_s* p, const float2* coeffs, float* xo, const float* wt, int batch, char* ws,
                     hipStream_t s) {
    const HostPlan& h = p->h;
    float2* W = reinterpret_cast<float2*>(ws);
    float2* Y = reinterpret_cast<float2*>(ws + align256(8 * h.C * batch));
    BigArgs a = big_args(p, ws, h.off_h_syn, h.spc ? h.spc : batch, false);
    a.cin = coeffs;
    a.W = W;
    a.wt = wt;
    if (int r = run_band_phase(p, false, coeffs, W, nullptr, wt, a, batch, s)) return r;
    if (int r = run_inv_a(p, W, Y, batch, s)) return r;
    return run_pass_b<true>(p, Y, reinterpret_cast<float2*>(xo), batch, static_cast<long long>(h.L), s);
}

// in_align / out_align: the alignment in bytes the kernels need of the input
// and output (8 for complex64 and for signals read or written in pairs, 4 for
// the sample-wise signal buffers of the sliced calls); the workspace needs 8.
int check_call(nsgcqt_plan_s* p, const void* in, const void* out, const void* ws, size_t ws_bytes,
               int64_t need, bool want_sliced, size_t in_align = 8, size_t out_align = 8) {
    if (!p) return set_err(NSGCQT_EINVAL, "plan is NULL");
    if (!in || !out) return set_err(NSGCQT_EINVAL, "input or output pointer is NULL");
    auto misaligned = [](const void* q, size_t a) { return (reinterpret_cast<uintptr_t>(q) & (a - 1)) != 0; };
    if (misaligned(in, in_align) || misaligned(out, out_align) || (ws && misaligned(ws, 8)))
        return set_err(NSGCQT_EINVAL, "input, output or workspace pointer is not aligned (" +
                                          std::to_string(in_align) + ", " + std::to_string(out_align) +
                                          " and 8 bytes)");
    if (p->h.sliced != want_sliced)
        return set_err(NSGCQT_EINVAL, want_sliced ? "plan is not a sliced plan" : "plan is a sliced plan");
    if (static_cast<int64_t>(ws_bytes) < need)
        return set_err(NSGCQT_EWORKSPACE, "workspace of " + std::to_string(ws_bytes) + " bytes, " +
                                              std::to_string(need) + " required");
    if (need > 0 && !ws) return set_err(NSGCQT_EINVAL, "workspace pointer is NULL");
    if (!p->device) return set_err(NSGCQT_EINVAL, "host-only plan has no device tables");
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != p->dev)
        return set_err(NSGCQT_EINVAL, "plan tables are on device " + std::to_string(p->dev) + ", device " +
                                          std::to_string(cur) + " is current");
    return NSGCQT_OK;
}

// Builds the host plan with `build(HostPlan&, std::string& err)` and, for a
// device plan, uploads its tables.
template <class Build>
int create(nsgcqt_plan* out, bool device, Build build) {
    if (!out) return set_err(NSGCQT_EINVAL, "out is NULL");
    *out = nullptr;
    nsgcqt_plan_s* p = new (std::nothrow) nsgcqt_plan_s();
    if (!p) return set_err(NSGCQT_ENOMEM, "host allocation failed");
    std::string err;
    int r;
    try {
        r = build(p->h, err);
    } catch (const std::bad_alloc&) {
        r = NSGCQT_ENOMEM;
        err = "host allocation failed while building the plan";
    } catch (const std::exception& ex) {
        r = NSGCQT_EINVAL;
        err = ex.what();
    }
    if (r != NSGCQT_OK) {
        delete p;
        return set_err(r, err);
    }
    schedule(p);
    if (device) {
        r = upload(p);
        if (r != NSGCQT_OK) {
            const std::string msg = g_err;
            release(p);
            delete p;
            return set_err(r, msg);
        }
    }
    *out = p;
    return NSGCQT_OK;
}

auto cq_builder(double fs, double fmin, double fmax, int bpo, int64_t n, int batch, bool sliced) {
    return [=](HostPlan& h, std::string& err) { return build_host_plan(h, fs, fmin, fmax, bpo, n, batch, sliced, err); };
}

int create_bands(nsgcqt_plan* out, double fs, int64_t n, int batch, int n_bands, const nsgcqt_band_spec* bands,
                 bool sliced, bool device) {
    if (out) *out = nullptr;
    if (n_bands < 1) return set_err(NSGCQT_EINVAL, "n_bands must be >= 1");
    if (!bands) return set_err(NSGCQT_EINVAL, "bands is NULL");
    std::vector<BandSpec> specs(n_bands);
    for (int i = 0; i < n_bands; ++i)
        specs[i] = BandSpec{bands[i].kind, bands[i].xi, bands[i].beta, bands[i].length, bands[i].centre_hz};
    return create(out, device, [&](HostPlan& h, std::string& err) {
        return build_host_plan_bands(h, fs, n, batch, specs, sliced, err);
    });
}

// Band count to *n and, with out non-NULL, the bands (capacity permitting).
int copy_specs(const std::vector<BandSpec>& specs, nsgcqt_band_spec* out, int capacity, int* n) {
    *n = static_cast<int>(specs.size());
    if (!out) return NSGCQT_OK;
    if (capacity < static_cast<int>(specs.size()))
        return set_err(NSGCQT_EINVAL, "capacity below the " + std::to_string(specs.size()) + " bands of the layout");
    for (size_t i = 0; i < specs.size(); ++i) {
        out[i].kind = specs[i].kind;
        out[i].xi = specs[i].xi;
        out[i].beta = specs[i].beta;
        out[i].length = specs[i].M;
        out[i].centre_hz = specs[i].f;
    }
    return NSGCQT_OK;
}

}  // namespace

extern "C" {

int nsgcqt_plan_create(nsgcqt_plan* out, double fs, double fmin, double fmax, int bpo, int64_t n, int batch) {
    return create(out, true, cq_builder(fs, fmin, fmax, bpo, n, batch, false));
}

int nsgcqt_plan_create_host(nsgcqt_plan* out, double fs, double fmin, double fmax, int bpo, int64_t n,
                            int batch) {
    return create(out, false, cq_builder(fs, fmin, fmax, bpo, n, batch, false));
}

int nsgcqt_sliced_plan_create(nsgcqt_plan* out, double fs, double fmin, double fmax, int bpo, int64_t slice_len,
                              int spc) {
    return create(out, true, cq_builder(fs, fmin, fmax, bpo, slice_len, spc, true));
}

int nsgcqt_sliced_plan_create_host(nsgcqt_plan* out, double fs, double fmin, double fmax, int bpo,
                                   int64_t slice_len, int spc) {
    return create(out, false, cq_builder(fs, fmin, fmax, bpo, slice_len, spc, true));
}

int nsgcqt_plan_create_bands(nsgcqt_plan* out, double fs, int64_t n_samples, int batch, int n_bands,
                             const nsgcqt_band_spec* bands) {
    return create_bands(out, fs, n_samples, batch, n_bands, bands, false, true);
}

int nsgcqt_plan_create_bands_host(nsgcqt_plan* out, double fs, int64_t n_samples, int batch, int n_bands,
                                  const nsgcqt_band_spec* bands) {
    return create_bands(out, fs, n_samples, batch, n_bands, bands, false, false);
}

int nsgcqt_sliced_plan_create_bands(nsgcqt_plan* out, double fs, int64_t slice_len, int slices_per_chunk,
                                    int n_bands, const nsgcqt_band_spec* bands) {
    return create_bands(out, fs, slice_len, slices_per_chunk, n_bands, bands, true, true);
}

int nsgcqt_sliced_plan_create_bands_host(nsgcqt_plan* out, double fs, int64_t slice_len, int slices_per_chunk,
                                         int n_bands, const nsgcqt_band_spec* bands) {
    return create_bands(out, fs, slice_len, slices_per_chunk, n_bands, bands, true, false);
}

int nsgcqt_layout_table1(nsgcqt_band_spec* out, int capacity, int* n_bands, double* fs, int64_t* n_samples) {
    if (!n_bands) return set_err(NSGCQT_EINVAL, "n_bands is NULL");
    std::vector<BandSpec> specs;
    table1_specs(specs);
    if (fs) *fs = kTable1Fs;
    if (n_samples) *n_samples = kTable1N;
    return copy_specs(specs, out, capacity, n_bands);
}

int nsgcqt_layout_erb(double fs, int64_t n_samples, double fmin, double fmax, double bands_per_erb,
                      nsgcqt_band_spec* out, int capacity, int* n_bands) {
    if (!n_bands) return set_err(NSGCQT_EINVAL, "n_bands is NULL");
    std::vector<BandSpec> specs;
    std::string err;
    try {
        if (int r = erb_specs(fs, n_samples, fmin, fmax, bands_per_erb, specs, err)) return set_err(r, err);
    } catch (const std::bad_alloc&) {
        return set_err(NSGCQT_ENOMEM, "host allocation failed");
    }
    if (specs.size() > static_cast<size_t>(INT32_MAX / 2)) return set_err(NSGCQT_EUNSUPPORTED, "too many bands");
    return copy_specs(specs, out, capacity, n_bands);
}

int nsgcqt_plan_destroy(nsgcqt_plan p) {
    if (!p) return NSGCQT_OK;
    const int r = release(p);
    delete p;
    return r;
}

int nsgcqt_plan_info(nsgcqt_plan p, nsgcqt_info* o) {
    if (!p || !o) return set_err(NSGCQT_EINVAL, "NULL argument");
    const HostPlan& h = p->h;
    std::memset(o, 0, sizeof(*o));
    o->n_bands = static_cast<int64_t>(h.bands.size());
    o->batch = h.batch;
    o->n_samples = h.N;
    o->packed_len = h.L;
    o->total_coeffs = h.C;
    o->max_band_len = h.maxM;
    o->max_fanout = h.max_fanout;
    o->max_overlap = h.max_overlap;
    o->sliced = h.sliced ? 1 : 0;
    o->ws_analyse = h.ws_an;
    o->ws_synthesise = h.ws_syn;
    o->ws_adjoint_analysis = h.ws_syn;
    o->ws_adjoint_synthesis = h.ws_an;
    o->table_bytes = p->dbytes;
    o->device_tables = p->device ? 1 : 0;
    return NSGCQT_OK;
}

int nsgcqt_band_info(nsgcqt_plan p, int band, nsgcqt_band* o) {
    if (!p || !o) return set_err(NSGCQT_EINVAL, "NULL argument");
    if (band < 0 || band >= static_cast<int>(p->h.bands.size()))
        return set_err(NSGCQT_EINVAL, "band index out of range");
    const HostBand& b = p->h.bands[band];
    o->kind = b.kind;
    o->k_lo = b.k_lo;
    o->k_hi = b.k_hi;
    o->k_centre = b.k_c;
    o->length = b.M;
    o->offset = b.off;
    o->centre_hz = b.f;
    o->xi = b.xi;
    o->beta = b.beta;
    const BandDev& d = p->h.banddev[band];
    o->fft_len = p->h.ffts[d.fft].n;
    o->bluestein = d.chirp >= 0 ? 1 : 0;
    return NSGCQT_OK;
}

int nsgcqt_plan_weights(nsgcqt_plan p, int which, float* dst, size_t bytes) {
    if (!p || !dst) return set_err(NSGCQT_EINVAL, "NULL argument");
    const std::vector<float>* v = nullptr;
    switch (which) {
        case 0: v = &p->h.wA; break;
        case 1: v = &p->h.wS; break;
        case 2: v = &p->h.wT; break;
        case 3: v = &p->h.wSa; break;
        default: return set_err(NSGCQT_EINVAL, "weight table index must be 0..3");
    }
    if (bytes < v->size() * sizeof(float)) return set_err(NSGCQT_EINVAL, "destination too small");
    std::memcpy(dst, v->data(), v->size() * sizeof(float));
    return NSGCQT_OK;
}

int nsgcqt_analyse(nsgcqt_plan p, const float* x, float* coeffs, void* ws, size_t ws_bytes, void* stream) {
    if (int r = check_call(p, x, coeffs, ws, ws_bytes, p ? p->h.ws_an : 0, false)) return r;
    std::lock_guard<std::mutex> lock(p->mu);
    p->ev_next = 0;
    return chain_analyse(p, x, reinterpret_cast<float2*>(coeffs), p->rA, p->h.batch, SliceIn{0, 0, 0, 0},
                         static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int nsgcqt_analyse_noalloc(nsgcqt_plan p, const float* x, float* coeffs, void* stream) {
    if (!p) return set_err(NSGCQT_EINVAL, "plan is NULL");
    if (p->h.ws_an > static_cast<int64_t>(NSGCQT_NOALLOC_SCRATCH_BYTES))
        return set_err(NSGCQT_EWORKSPACE, "the plan's analysis needs " + std::to_string(p->h.ws_an) +
                                              " bytes of workspace, the allocation-free analysis has " +
                                              std::to_string(NSGCQT_NOALLOC_SCRATCH_BYTES));
    if (!p->device) return set_err(NSGCQT_EINVAL, "host-only plan has no device tables");
    void* ws = nullptr;
    if (int r = scratch_address(&ws)) return r;
    if (int r = check_call(p, x, coeffs, ws, NSGCQT_NOALLOC_SCRATCH_BYTES, p->h.ws_an, false)) return r;
    std::lock_guard<std::mutex> lock(p->mu);
    p->ev_next = 0;
    return chain_analyse(p, x, reinterpret_cast<float2*>(coeffs), p->rA, p->h.batch, SliceIn{0, 0, 0, 0},
                         static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int nsgcqt_synthesise(nsgcqt_plan p, const float* coeffs, float* xo, void* ws, size_t ws_bytes, void* stream) {
    if (int r = check_call(p, coeffs, xo, ws, ws_bytes, p ? p->h.ws_syn : 0, false)) return r;
    std::lock_guard<std::mutex> lock(p->mu);
    p->ev_next = 0;
    return chain_synthesise(p, reinterpret_cast<const float2*>(coeffs), xo, p->wS, p->h.batch,
                            static_cast<char*>(ws), static_cast<hipStream_t>(stream));
}

int nsgcqt_adjoint(nsgcqt_plan p, int op, const float* in, float* out, void* ws, size_t ws_bytes, void* stream) {
    if (op != NSGCQT_OP_ADJ_ANALYSIS && op != NSGCQT_OP_ADJ_SYNTHESIS)
        return set_err(NSGCQT_EINVAL, "op must be NSGCQT_OP_ADJ_ANALYSIS or NSGCQT_OP_ADJ_SYNTHESIS");
    const bool ta = op == NSGCQT_OP_ADJ_ANALYSIS;
    if (int r = check_call(p, in, out, ws, ws_bytes, p ? (ta ? p->h.ws_syn : p->h.ws_an) : 0, false)) return r;
    std::lock_guard<std::mutex> lock(p->mu);
    p->ev_next = 0;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (ta)
        return chain_synthesise(p, reinterpret_cast<const float2*>(in), out, p->wT, p->h.batch,
                                static_cast<char*>(ws), s);
    return chain_analyse(p, in, reinterpret_cast<float2*>(out), p->rSa, p->h.batch, SliceIn{0, 0, 0, 0},
                         static_cast<char*>(ws), s);
}

int64_t nsgcqt_sliced_count(nsgcqt_plan p, int64_t n) {
    if (!p || !p->h.sliced) return set_err(NSGCQT_EINVAL, "not a sliced plan");
    if (n < 0) return set_err(NSGCQT_EINVAL, "negative length");
    const int64_t H = p->h.N / 2;
    return (n + H - 1) / H + 1;
}

int nsgcqt_sliced_analyse(nsgcqt_plan p, const float* x, int64_t n, float* coeffs, void* ws, size_t ws_bytes,
                          void* stream) {
    if (int r = check_call(p, x, coeffs, ws, ws_bytes, p ? p->h.ws_an : 0, true, 4, 8)) return r;
    if (n < 1) return set_err(NSGCQT_EINVAL, "signal length must be >= 1");
    std::lock_guard<std::mutex> lock(p->mu);
    const HostPlan& h = p->h;
    const int64_t J = nsgcqt_sliced_count(p, n);
    hipStream_t s = static_cast<hipStream_t>(stream);
    p->ev_next = 0;
    for (int64_t s0 = 0; s0 < J; s0 += h.spc) {
        const int cnt = static_cast<int>(std::min<int64_t>(h.spc, J - s0));
        SliceIn sl{1, static_cast<int>(s0), static_cast<long long>(n), static_cast<int>(h.N / 2)};
        float2* c = reinterpret_cast<float2*>(coeffs) + s0 * h.C;
        if (int r = chain_analyse(p, x, c, p->rA, cnt, sl, static_cast<char*>(ws), s)) return r;
    }
    return NSGCQT_OK;
}

int nsgcqt_sliced_synthesise(nsgcqt_plan p, const float* coeffs, int64_t n, float* xo, void* ws,
                             size_t ws_bytes, void* stream) {
    if (int r = check_call(p, coeffs, xo, ws, ws_bytes, p ? p->h.ws_syn : 0, true, 8, 4)) return r;
    if (n < 1) return set_err(NSGCQT_EINVAL, "signal length must be >= 1");
    std::lock_guard<std::mutex> lock(p->mu);
    const HostPlan& h = p->h;
    const int64_t J = nsgcqt_sliced_count(p, n);
    const int64_t H = h.N / 2;
    char* w = static_cast<char*>(ws);
    const int64_t chain_bytes = h.off_y_sliced;
    float* y = reinterpret_cast<float*>(w + chain_bytes);
    float* carry[2] = {reinterpret_cast<float*>(w + chain_bytes + align256(4 * h.N * h.spc)),
                       reinterpret_cast<float*>(w + chain_bytes + align256(4 * h.N * h.spc) + align256(4 * H))};
    hipStream_t s = static_cast<hipStream_t>(stream);
    p->ev_next = 0;
    int flip = 0;
    for (int64_t s0 = 0; s0 < J; s0 += h.spc) {
        const int cnt = static_cast<int>(std::min<int64_t>(h.spc, J - s0));
        const float2* c = reinterpret_cast<const float2*>(coeffs) + s0 * h.C;
        if (int r = chain_synthesise(p, c, y, p->wS, cnt, w, s)) return r;
        const int64_t span = static_cast<int64_t>(cnt) * H;
        const int blocks = static_cast<int>(std::min<int64_t>((span + 255) / 256, 8192));
        ev_start(p, s);
        LAUNCH_TRY(k_ola, dim3(blocks), dim3(256), 0, s, y, carry[flip], carry[flip ^ 1], xo,
                   static_cast<int>(s0), cnt, static_cast<int>(h.N), static_cast<long long>(n));
        ev_end(p, s);
        flip ^= 1;
    }
    return NSGCQT_OK;
}

int nsgcqt_set_stage_events(nsgcqt_plan p, void* const* events, int n_events) {
    if (!p) return set_err(NSGCQT_EINVAL, "plan is NULL");
    std::lock_guard<std::mutex> lock(p->mu);
    p->events.clear();
    p->ev_next = 0;
    if (events && n_events > 0)
        for (int i = 0; i < n_events; ++i) p->events.push_back(static_cast<hipEvent_t>(events[i]));
    return NSGCQT_OK;
}

int nsgcqt_stage_info(nsgcqt_plan p, int op, int i, char* name, size_t cap, double* alg_bytes) {
    if (!p) return set_err(NSGCQT_EINVAL, "plan is NULL");
    if (op < 0 || op > 3) return set_err(NSGCQT_EINVAL, "unknown op");
    const HostPlan& h = p->h;
    // a sliced plan lists the kernels of one chunk of h.batch (= slices per
    // chunk) slices: the analysis chain, or the synthesis chain and the
    // overlap-add of the chunk's slices
    if (h.sliced && op != NSGCQT_OP_ANALYSE && op != NSGCQT_OP_SYNTHESISE)
        return set_err(NSGCQT_EINVAL, "a sliced plan runs analysis and synthesis only");
    const double b = h.batch, L = static_cast<double>(h.L), C = static_cast<double>(h.C);
    struct St { std::string name; double bytes; };
    std::vector<St> st;
    const bool an = (op == NSGCQT_OP_ANALYSE || op == NSGCQT_OP_ADJ_SYNTHESIS);
    if (an) {
        st.push_back({"fft_fwd_a", 16.0 * L * b});
        st.push_back({"fft_fwd_b", 16.0 * L * b});
    }
    // huge-band passes: the column pass reads its input share and writes the
    // intermediate, the row pass reads it and writes the output or the
    // Bluestein midpoint
    const double hn = static_cast<double>(h.Hn), hb = static_cast<double>(h.Hn_blu), cg = static_cast<double>(h.C_big);
    std::vector<St> big;
    if (!h.bigs.empty()) {
        const double in0 = an ? cg / C * 8.0 * L : 8.0 * cg;
        big.push_back({an ? "big_analysis_a" : "big_synthesis_a", (in0 + 8.0 * hn) * b});
        const double cbb = static_cast<double>(h.C_big_blu);
        big.push_back({an ? "big_analysis_b" : "big_synthesis_b", (8.0 * hn + 8.0 * (cg - cbb) + 8.0 * hb) * b});
        if (h.big_n[2]) {
            big.push_back({an ? "big_analysis_a2" : "big_synthesis_a2", 16.0 * hb * b});
            big.push_back({an ? "big_analysis_b2" : "big_synthesis_b2", (8.0 * hb + 8.0 * cbb) * b});
        }
    }
    // the band phase in launch order
    for (int u : p->order) {
        if (u == static_cast<int>(h.buckets.size())) {
            st.insert(st.end(), big.begin(), big.end());
            continue;
        }
        const Bucket& bk = h.buckets[u];
        const double cb = static_cast<double>(bk.coeffs);
        const std::string shape = std::to_string(bk.nt) + "x" + std::to_string(bk.ept);
        if (an) st.push_back({"band_analysis_" + shape, (cb / C * 8.0 * L + 8.0 * cb) * b});
        else st.push_back({"band_synthesis_" + shape, 16.0 * cb * b});
    }
    if (!an) {
        st.push_back({"fft_inv_a_overlap_add", (8.0 * C + 8.0 * L) * b});
        st.push_back({"fft_inv_b", 16.0 * L * b});
        // per slice: read its N synthesised samples, write the H = N / 2
        // output samples it completes
        if (h.sliced) st.push_back({"sliced_overlap_add", 6.0 * static_cast<double>(h.N) * b});
    }
    if (i >= 0 && i < static_cast<int>(st.size())) {
        if (name && cap) {
            std::strncpy(name, st[i].name.c_str(), cap - 1);
            name[cap - 1] = 0;
        }
        if (alg_bytes) *alg_bytes = st[i].bytes;
    }
    return static_cast<int>(st.size());
}

const char* nsgcqt_last_error(void) { return g_err.c_str(); }

}  // extern "C"
