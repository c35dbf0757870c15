// Runs the plan kernels' own source on the CPU, under AddressSanitizer and
// UndefinedBehaviorSanitizer: workgroups one at a time, one fiber per work-item, a
// real workgroup barrier and exec-masked wave exchanges (ballot, DPP).  LDS starts
// every workgroup filled with garbage, and every output array is an allocation of its
// own, so a read of LDS before it is written or an access outside an array shows.
//
// The plan arguments come from the library's host code (plan_args, the same code the
// C entry point runs).  Input file: L N C, per level H W scale, finest_scale, K,
// box_convention, then K RoIs of 5 floats.  Output file: the tile layout, the levels,
// offsets, keys, permutation and tile lists (written at the end of main).
#include "hip/hip_runtime.h"

#include <sanitizer/common_interface_defs.h>
#include <sys/mman.h>
#include <ucontext.h>

#include <fstream>
#include <functional>

thread_local EmuDim threadIdx;
EmuDim blockIdx, blockDim, gridDim;
int32_t *emu_smem;
static std::vector<std::pair<void *, size_t>> g_reg;   // the kernels' static LDS arrays

// Every work-item registers the static LDS arrays of its kernel before touching them;
// the first registration fills the array with garbage (later workgroups get theirs
// from launch()).
void emu_register(void *p, size_t n) {
    for (auto &r : g_reg)
        if (r.first == p) return;
    std::memset(p, 0x5a, n);
    g_reg.push_back({p, n});
}

// Work-items are fibers on one host thread (ucontext), switched only at the points
// where they wait for each other: the workgroup barrier and the wave exchanges.  After
// every runnable work-item has run to its next wait, the waves whose lanes all wait
// (or have finished) complete their exchange, an exchange taking the lanes that reached
// it (the others are inactive, as under an exec mask); when no exchange is pending and
// every work-item waits at the barrier or has finished, the barrier opens.
enum { kReady, kBarrier, kExchange, kDone };
struct Fiber {
    ucontext_t ctx;
    int state;
    int val;
};
struct Wave {
    int val[64];
    bool act[64];
};
static ucontext_t g_main;
static std::vector<Fiber> g_fib;
static std::vector<Wave> g_wave;
static int g_cur;
static const void *g_main_bottom;
static size_t g_main_size;
static char *g_stacks;
// Each fiber's stack sits above a page that faults on access, so an overflow ends the
// run instead of writing into the next stack.  (The sanitizer clears the shadow of the
// whole stack at every switch: a small stack keeps switches cheap.)
constexpr size_t kGuard = 4096;
constexpr size_t kStack = 64 * 1024;
constexpr int kMaxItems = 1024;
static char *stack_of(int i) { return g_stacks + (kGuard + kStack) * i + kGuard; }
static std::function<void()> g_kern;

static void to_main(bool done) {
    void *fake = nullptr;
    __sanitizer_start_switch_fiber(done ? nullptr : &fake, g_main_bottom, g_main_size);
    if (done) return;   // the fiber returns to uc_link
    swapcontext(&g_fib[g_cur].ctx, &g_main);
    __sanitizer_finish_switch_fiber(fake, &g_main_bottom, &g_main_size);
    threadIdx.x = g_cur;
}

static void fiber_entry() {
    __sanitizer_finish_switch_fiber(nullptr, &g_main_bottom, &g_main_size);
    threadIdx.x = g_cur;
    g_kern();
    g_fib[g_cur].state = kDone;
    to_main(true);
}

static void wait_at(int state) {
    g_fib[g_cur].state = state;
    to_main(false);
}

void __syncthreads() { wait_at(kBarrier); }

static int wave_xchg(int v, const int *&vals, const bool *&act) {
    g_fib[g_cur].val = v;
    wait_at(kExchange);
    const Wave &w = g_wave[g_cur >> 6];
    vals = w.val;
    act = w.act;
    return g_cur & 63;
}

unsigned long long __ballot(int pred) {
    const int *vals;
    const bool *act;
    wave_xchg(pred != 0, vals, act);
    unsigned long long m = 0;
    for (int i = 0; i < 64; ++i)
        if (act[i] && vals[i]) m |= 1ull << i;
    return m;
}

// Runs one workgroup of n work-items to completion.
static void run_block(int n) {
    if (!g_stacks) {
        const size_t bytes = (kGuard + kStack) * kMaxItems;
        g_stacks = static_cast<char *>(mmap(nullptr, bytes, PROT_READ | PROT_WRITE,
                                            MAP_PRIVATE | MAP_ANONYMOUS, -1, 0));
        if (g_stacks == MAP_FAILED) std::abort();
        for (int i = 0; i < kMaxItems; ++i)
            if (mprotect(stack_of(i) - kGuard, kGuard, PROT_NONE) != 0) std::abort();
    }
    if (n > kMaxItems) std::abort();
    g_fib.assign(n, Fiber{});
    g_wave.assign((n + 63) / 64, Wave{});
    for (int i = 0; i < n; ++i) {
        Fiber &f = g_fib[i];
        getcontext(&f.ctx);
        f.ctx.uc_stack.ss_sp = stack_of(i);
        f.ctx.uc_stack.ss_size = kStack;
        f.ctx.uc_link = &g_main;
        makecontext(&f.ctx, fiber_entry, 0);
        f.state = kReady;
    }
    for (;;) {
        bool ran = false;
        for (int i = 0; i < n; ++i) {
            if (g_fib[i].state != kReady) continue;
            ran = true;
            g_cur = i;
            void *fake = nullptr;
            __sanitizer_start_switch_fiber(&fake, stack_of(i), kStack);
            swapcontext(&g_main, &g_fib[i].ctx);
            __sanitizer_finish_switch_fiber(fake, nullptr, nullptr);
        }
        bool exchanged = false;
        for (int w = 0; w * 64 < n; ++w) {
            const int lo = w * 64, hi = std::min(n, lo + 64);
            bool any = false, all = true;
            for (int i = lo; i < hi; ++i) {
                any |= g_fib[i].state == kExchange;
                all &= g_fib[i].state != kReady;
            }
            if (!any || !all) continue;
            Wave &x = g_wave[w];
            for (int i = lo; i < lo + 64; ++i) {
                const bool a = i < hi && g_fib[i].state == kExchange;
                x.act[i - lo] = a;
                x.val[i - lo] = a ? g_fib[i].val : 0;
                if (a) g_fib[i].state = kReady;
            }
            exchanged = true;
        }
        if (exchanged) continue;
        int waiting = 0, done = 0;
        for (auto &f : g_fib) {
            waiting += f.state == kBarrier;
            done += f.state == kDone;
        }
        if (done == n) return;
        if (waiting + done == n) {
            for (auto &f : g_fib)
                if (f.state == kBarrier) f.state = kReady;
            continue;
        }
        if (!ran) {
            std::printf("deadlock: work-items wait for each other\n");
            std::abort();
        }
    }
}

// DPP moves: row_shr:n (0x111..0x11f) within each row of 16 lanes, row_bcast:15
// (0x142) and row_bcast:31 (0x143).  A read of an inactive lane aborts.
int emu_update_dpp(int old, int src, int ctrl, int row_mask, int, bool bound) {
    const int *vals;
    const bool *act;
    const int l = wave_xchg(src, vals, act), row = l >> 4;
    if (!((row_mask >> row) & 1)) return old;
    int s = -1;
    if (ctrl >= 0x111 && ctrl <= 0x11f) {
        const int n = ctrl - 0x110;
        if ((l & 15) >= n) s = l - n;
    } else if (ctrl == 0x142) {
        if (row >= 1) s = row * 16 - 1;
    } else if (ctrl == 0x143) {
        if (row >= 2) s = 31;
    } else {
        std::printf("DPP control %x not emulated\n", ctrl);
        std::abort();
    }
    if (s >= 0 && !act[s]) {
        std::printf("DPP reads an inactive lane\n");
        std::abort();
    }
    return s >= 0 ? vals[s] : (bound ? 0 : old);
}

template <typename F> static void launch(int grid, int threads, size_t smem_words, F &&kern) {
    gridDim.x = grid;
    blockDim.x = threads;
    g_kern = kern;
    for (int b = 0; b < grid; ++b) {
        blockIdx.x = b;
        for (auto &r : g_reg) std::memset(r.first, 0x5a, r.second);
        emu_smem = smem_words ? static_cast<int32_t *>(std::malloc(smem_words * 4)) : nullptr;
        if (emu_smem) std::memset(emu_smem, 0x5a, smem_words * 4);
        run_block(threads);
        std::free(emu_smem);
        emu_smem = nullptr;
    }
}

// The kernels (plan.hip without its launchers, generated) and the host code.
#include "plan_kernels.inc"
#include "api.hip"

hipError_t hipGetDevice(int *d) {
    *d = 0;
    return hipSuccess;
}
static unsigned char g_symbol[1 << 20];
hipError_t hipGetSymbolAddress(void **p, const void *) {
    *p = g_symbol;
    return hipSuccess;
}
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t n, hipMemcpyKind, hipStream_t) {
    std::memmove(dst, src, n);
    return hipSuccess;
}

namespace rex {
static bool g_force_multi = false;

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t box_plus1, int32_t *out, hipStream_t) {
    launch(std::max(1, std::min((K + 255) / 256, 4096)), 256, 0,
           [&] { level_map_kernel(rois, K, L, finest_scale, box_plus1, out); });
    return hipSuccess;
}

// The launch sequence of the library's launch_plan.
hipError_t launch_plan(const PlanArgs &a, hipStream_t) {
    const int words = plan_one_words(a);
    if (!g_force_multi && a.K <= kPlanOne && words <= kPlanWords &&
        (a.ntiles <= 0 || a.nbands > 0)) {
        launch(a.ntiles > 0 ? 2 + a.nbands : 1, kPlanThreads, words, [&] { plan_one_kernel(a); });
        return hipSuccess;
    }
    launch(std::max(1, std::min((a.nbins + 255) / 256, 1024)), 256, 0,
           [&] { plan_clear_kernel(a.key_count, a.nbins); });
    launch(std::max(1, std::min((a.K + 255) / 256, 4096)), 256, 0, [&] { plan_count_kernel(a); });
    launch(1, kPlanThreads, a.nbins + kPlanThreads, [&] { plan_scan_kernel(a); });
    launch(std::max(1, std::min((a.K + 15) / 16, 4096)), 256, 0, [&] { plan_fill_kernel(a); });
    if (a.ntiles > 0) launch(1, kPlanThreads, 0, [&] { plan_order_kernel(a); });
    return hipSuccess;
}

// Not run by the emulator.
bool fwd_fast_available(int, int, int) { return false; }
bool bwd_fast_available(int, int, int) { return false; }
bool gather_available(int, int, int) { return false; }
bool pool_fwd_fast_available(int, int) { return false; }
bool pool_gather_available(int, int) { return false; }
hipError_t launch_fwd(FwdArgs, int, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_fwd_multi(FwdMultiArgs, int, int, hipStream_t) { std::abort(); }
hipError_t launch_bwd(BwdArgs, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_gather(GatherArgs, int, hipStream_t) { std::abort(); }
hipError_t launch_zero(const LevelTable &, const int64_t *, const int *, hipStream_t) { std::abort(); }
hipError_t launch_pool_fwd(PoolArgs, int, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_pool_bwd(PoolArgs, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_pool_gather(GatherArgs, int, hipStream_t) { std::abort(); }
hipError_t launch_deform_fwd(DeformArgs, int, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_deform_bwd(DeformArgs, int, int, bool, hipStream_t) { std::abort(); }
hipError_t launch_deform_gather(GatherArgs, const DeformArgs &, int, hipStream_t) { std::abort(); }
bool deform_gather_available(int, int, int) { return false; }
hipError_t launch_nms(NmsArgs, hipStream_t) { std::abort(); }
hipError_t launch_nms_batched(const NmsBatchArgs &, hipStream_t) { std::abort(); }
}  // namespace rex

template <typename T> static T *array(size_t n, std::vector<void *> &all) {
    const size_t m = std::max<size_t>(n, 1);
    T *p = static_cast<T *>(std::malloc(m * sizeof(T)));
    std::memset(p, 0x7f, m * sizeof(T));
    all.push_back(p);
    return p;
}

template <typename T> static void put(std::ofstream &o, const T *p, size_t n) {
    o.write(reinterpret_cast<const char *>(p), static_cast<std::streamsize>(n * sizeof(T)));
}

int main(int argc, char **argv) {
    if (argc < 3) {
        std::printf("usage: emu input output [multi]\n");
        return 2;
    }
    rex::g_force_multi = argc > 3;
    std::ifstream f(argv[1], std::ios::binary);
    int32_t L, N, C;
    f.read(reinterpret_cast<char *>(&L), 4);
    f.read(reinterpret_cast<char *>(&N), 4);
    f.read(reinterpret_cast<char *>(&C), 4);
    rex::LevelTable t{};
    t.num = L;
    t.N = N;
    t.C = C;
    for (int l = 0; l < L; ++l) {
        f.read(reinterpret_cast<char *>(&t.l[l].H), 4);
        f.read(reinterpret_cast<char *>(&t.l[l].W), 4);
        f.read(reinterpret_cast<char *>(&t.l[l].scale), 4);
    }
    float fs;
    int32_t K, conv;
    f.read(reinterpret_cast<char *>(&fs), 4);
    f.read(reinterpret_cast<char *>(&K), 4);
    f.read(reinterpret_cast<char *>(&conv), 4);
    std::vector<void *> all;
    float *rois = array<float>(5 * size_t(K), all);
    f.read(reinterpret_cast<char *>(rois), 20 * std::streamsize(K));
    int32_t *lv = array<int32_t>(K, all);

    const rex::TileLayout tl = tile_layout(t, K);
    rex::PlanArgs a{};
    static char ws_base[256];   // the workspace pointers are replaced below
    if (plan_args(t, rois, K, fs, conv, lv, ws_base, tl, &a) != RE_OK) {
        std::printf("plan_args refused the input\n");
        return 3;
    }
    a.offsets = array<int32_t>(L + 1, all);
    a.perm = array<int32_t>(K, all);
    a.keys = array<int32_t>(K, all);
    a.tile_start = array<int32_t>(a.ntiles, all);
    a.tile_end = array<int32_t>(a.ntiles, all);
    a.tile_order = array<int32_t>(a.ntiles, all);
    a.tile_rois = array<int32_t>(a.capacity, all);
    a.key_count = array<int32_t>(rex::kPlanMaxBins, all);
    std::printf("K %d ntiles %d nbands %d capacity %d path %s\n", K, a.ntiles, a.nbands,
                a.capacity, rex::g_force_multi ? "multi" : "auto");
    rex::launch_plan(a, nullptr);

    // header: ntiles capacity K L tile_shift ntx[8] nty[8] tbase[9]
    std::ofstream o(argv[2], std::ios::binary);
    const int32_t hdr[5] = {a.ntiles, a.capacity, K, L, a.tile_shift};
    put(o, hdr, 5);
    put(o, a.ntx, rex::kMaxLevels);
    put(o, a.nty, rex::kMaxLevels);
    put(o, a.tbase, rex::kMaxLevels + 1);
    put(o, lv, K);
    put(o, a.offsets, L + 1);
    put(o, a.keys, K);
    put(o, a.perm, K);
    put(o, a.tile_start, a.ntiles);
    put(o, a.tile_end, a.ntiles);
    put(o, a.tile_order, a.ntiles);
    put(o, a.tile_rois, size_t(a.capacity));
    for (void *p : all) std::free(p);
    std::printf("done\n");
    return 0;
}
