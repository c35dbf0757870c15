// select.hip -- per-category proposal selection: greedy NMS or Soft-NMS.
//
// A two-stage detector turns each image's (or class's) scored boxes into proposals
// with NMS; the paper runs its bbox operations on the GPU (§1) and lists Soft-NMS
// among its general modules (§2).  One call selects within every category of a batch:
// one category per image (or class), each category independent.  Definition (candidate
// rule, rank order, decay, dropping, ties) in include/roi_extract.h.
//
// Kernels on one stream:
//   nmsb_clear_kernel    zero the per-category counters
//   nmsb_count_kernel    candidates per category (score >= threshold, valid category)
//   nmsb_scan_kernel     one workgroup: category starts (exclusive scan) and cursors
//   nmsb_place_kernel    every candidate to a slot of its category's range
//   nmsb_select_kernel   one 1024-thread workgroup per category (grid-stride over the
//                        categories): sorts the category's candidates by rank (bitonic
//                        network in LDS, or in global memory above kSegLds candidates),
//                        then either walks them in blocks of 64 against the growing list
//                        of kept boxes (greedy NMS: the 16 waves test a block against
//                        the kept list in parallel, wave 0 resolves the block's own
//                        overlaps in order), or runs Soft-NMS (each iteration decays the
//                        remaining candidates against the last selected box and selects
//                        the largest current score with a workgroup min-reduction of a
//                        64-bit key: score rank key above the rank position).
#include "internal.hpp"

namespace rex {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSegLds = 8192;    // candidates a category sorts in LDS (64 KiB of keys)
constexpr int kSoftReg = 4;      // Soft-NMS candidates per thread held in registers
constexpr int kSoftLdsBoxes = 3072;   // Soft-NMS: categories up to this size keep boxes in LDS

__global__ __launch_bounds__(256) void nmsb_clear_kernel(int32_t *count, int32_t n) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        count[i] = 0;
}

__device__ __forceinline__ int nmsb_category(const NmsBatchArgs &a, int32_t i) {
    const int c = a.categories ? a.categories[i] : 0;
    // a candidate: a category of the batch and a score at or above the threshold (a NaN
    // score never is)
    return (c >= 0 && c < a.C && a.scores[i] >= a.score_threshold) ? c : -1;
}

// Candidate counting and placement work on contiguous ranges of kPlaceRange boxes per
// workgroup: the workgroup counts its boxes per category in LDS and touches each
// category's device counter once.  Device-scope atomics to one address are serialised
// beyond the per-XCD L2 (about 0.2 us each), so one per box and category -- thousands
// on each of a few counters -- would dominate the selection.
constexpr int kPlaceThreads = 256;
constexpr int kPlaceRange = 4096;

__device__ __forceinline__ void nmsb_range(const NmsBatchArgs &a, int32_t &i0, int32_t &i1) {
    i0 = static_cast<int32_t>(blockIdx.x) * kPlaceRange;
    i1 = min(a.N, i0 + kPlaceRange);
}

__global__ __launch_bounds__(kPlaceThreads) void nmsb_count_kernel(NmsBatchArgs a) {
    extern __shared__ int32_t hist[];   // [C]
    for (int c = threadIdx.x; c < a.C; c += kPlaceThreads) hist[c] = 0;
    __syncthreads();
    int32_t i0, i1;
    nmsb_range(a, i0, i1);
    for (int32_t i = i0 + threadIdx.x; i < i1; i += kPlaceThreads) {
        const int c = nmsb_category(a, i);
        if (c >= 0) atomicAdd(&hist[c], 1);
    }
    __syncthreads();
    for (int c = threadIdx.x; c < a.C; c += kPlaceThreads)
        if (hist[c] > 0) atomicAdd(&a.count[c], hist[c]);
}

__global__ __launch_bounds__(kSelThreads) void nmsb_scan_kernel(NmsBatchArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;              // [C]
    int32_t *part = smem + a.C;        // scan scratch
    for (int i = threadIdx.x; i < a.C; i += kSelThreads) hist[i] = a.count[i];
    __syncthreads();
    const int total = block_exclusive_scan(hist, a.C, part);
    for (int i = threadIdx.x; i < a.C; i += kSelThreads) {
        a.start[i] = hist[i];
        a.count[i] = hist[i];   // becomes the placement cursor
    }
    if (threadIdx.x == 0) a.start[a.C] = total;
}

// Every candidate of the workgroup's range to a slot of its category: the range's count
// per category reserves a run of slots with one device atomic, then LDS cursors deal the
// run out.  The order inside a category is free (the selection sorts it).
__global__ __launch_bounds__(kPlaceThreads) void nmsb_place_kernel(NmsBatchArgs a) {
    extern __shared__ int32_t cur[];   // [C]: counts, then cursors
    for (int c = threadIdx.x; c < a.C; c += kPlaceThreads) cur[c] = 0;
    __syncthreads();
    int32_t i0, i1;
    nmsb_range(a, i0, i1);
    for (int32_t i = i0 + threadIdx.x; i < i1; i += kPlaceThreads) {
        const int c = nmsb_category(a, i);
        if (c >= 0) atomicAdd(&cur[c], 1);
    }
    __syncthreads();
    for (int c = threadIdx.x; c < a.C; c += kPlaceThreads)
        if (cur[c] > 0) cur[c] = atomicAdd(&a.count[c], cur[c]);
    __syncthreads();
    for (int32_t i = i0 + threadIdx.x; i < i1; i += kPlaceThreads) {
        const int c = nmsb_category(a, i);
        if (c < 0) continue;
        const int slot = atomicAdd(&cur[c], 1);
        if (slot >= 0 && slot < a.N) a.sidx[slot] = i;
    }
}

// Gaussian decay weight exp(-iou^2 / sigma) rounded to binary32.  exp is evaluated in
// double by scaling and squaring: the argument is halved until it lies in [-1/2, 0], a
// degree-16 Taylor polynomial is summed in Horner form, and the result is squared back;
// every double operation is rounded once, in the written order, so the weight -- which
// decides the next selection -- does not depend on the machine's exp.  Below -128 the
// exponential rounds to +0.
__device__ __forceinline__ float soft_gauss_weight(float iou, float sigma) {
    if (!(iou > 0.0f)) return 1.0f;
    double x = -(static_cast<double>(iou) * static_cast<double>(iou)) / static_cast<double>(sigma);
    if (!(x >= -128.0)) return 0.0f;
    int k = 0;
    while (x < -0.5) {
        x = x * 0.5;
        ++k;
    }
    double e = 1.0;
    for (int n = 16; n >= 1; --n) e = 1.0 + (x * e) / static_cast<double>(n);
    for (int i = 0; i < k; ++i) e = e * e;
    return static_cast<float>(e);
}

// New current score of a candidate after the box `m` was selected; NaN IoU: unchanged.
__device__ __forceinline__ float soft_decay(const NmsBatchArgs &a, float4 m, float4 b, float s) {
    const float iou = nms_iou(m, b);
    if (iou != iou) return s;
    if (a.method == kNmsLinear) {
        if (iou > a.iou_threshold) {
            const float w = 1.0f - iou;
            s = s * w;
        }
        return s;
    }
    return s * soft_gauss_weight(iou, a.sigma);
}

// Ascending sort of keys[0, n) with every position >= n taken as +infinity: the bitonic
// network in the form whose every comparator puts the smaller key at the lower position
// (each merge stage starts by comparing a position with its mirror in the block, then
// halves), so a comparator with its partner past n is a no-op and any n works.  Called
// by the whole workgroup; `keys` in LDS or global memory (sync after every stage).
template <typename Ptr>
__device__ void bitonic_sort_n(Ptr keys, int n) {
    int P = 1;
    while (P < n) P <<= 1;
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int q = threadIdx.x; q < P / 2; q += kSelThreads) {
                int i, p;
                if (j == (k >> 1)) {   // mirror step
                    i = (q / j) * k + (q % j);
                    p = i ^ (k - 1);
                } else {
                    i = ((q & ~(j - 1)) << 1) | (q & (j - 1));
                    p = i + j;
                }
                if (p < n) {
                    const uint64_t x = keys[i], y = keys[p];
                    if (x > y) {
                        keys[i] = y;
                        keys[p] = x;
                    }
                }
            }
            __syncthreads();
        }
    }
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t w = __shfl_xor(v, o, 64);
        v = w < v ? w : v;
    }
    return v;
}

// Greedy NMS over the sorted candidates [base, base + n) of category c.
__device__ void select_greedy(const NmsBatchArgs &a, int c, int base, int n, uint64_t *lds) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float4 *cand = reinterpret_cast<float4 *>(lds);                    // [64] the block
    unsigned long long *hit = reinterpret_cast<unsigned long long *>(cand + 64);   // [1]
    int32_t *s_kept = reinterpret_cast<int32_t *>(hit + 1);            // [1]
    const int limit = a.max_keep;
    int kept = 0;
    for (int b0 = 0; b0 < n && kept < limit; b0 += 64) {
        const int nb = min(64, n - b0);
        if (tid < 64 && tid < nb) cand[tid] = a.sbox[base + b0 + tid];
        if (tid == 0) *hit = 0;
        __syncthreads();
        // every wave tests the block against its share of the kept list
        {
            const float4 mine = lane < nb ? cand[lane] : make_float4(0, 0, 0, 0);
            bool h = false;
            for (int k = wave; k < kept; k += kSelWaves) {
                const float4 kb = a.kbox[base + k];
                h = h || (nms_iou(kb, mine) > a.iou_threshold);
            }
            const uint64_t bits = __ballot(h && lane < nb);
            if (lane == 0 && bits) atomicOr(hit, static_cast<unsigned long long>(bits));
        }
        __syncthreads();
        if (wave == 0) {
            // the block's own overlaps: bit u of lane t marks a later candidate u of the
            // block that candidate t removes
            uint64_t dbits = 0;
            if (lane < nb) {
                const float4 mine = cand[lane];
                for (int u = lane + 1; u < nb; ++u)
                    if (nms_iou(mine, cand[u]) > a.iou_threshold) dbits |= uint64_t(1) << u;
            }
            const uint64_t h0 = *hit;
            uint64_t rem = (static_cast<uint64_t>(static_cast<uint32_t>(
                                __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(h0 >> 32))))
                            << 32) |
                           static_cast<uint32_t>(
                               __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(h0)));
            uint64_t keptm = 0;
            int nk = kept;
            for (int t = 0; t < nb && nk < limit; ++t) {
                if (!((rem >> t) & 1)) {
                    keptm |= uint64_t(1) << t;
                    ++nk;
                    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(dbits), t);
                    const uint32_t hi =
                        __builtin_amdgcn_readlane(static_cast<uint32_t>(dbits >> 32), t);
                    rem |= (static_cast<uint64_t>(hi) << 32) | lo;
                }
            }
            if ((keptm >> lane) & 1) {
                const int r = kept + __popcll(keptm & ((uint64_t(1) << lane) - 1));
                const int pos = base + b0 + lane;
                a.kbox[base + r] = cand[lane];
                a.keep[static_cast<int64_t>(c) * limit + r] = a.sidx[pos];
                a.kept_scores[static_cast<int64_t>(c) * limit + r] = a.sscore[pos];
            }
            if (lane == 0) *s_kept = nk;
        }
        __syncthreads();
        kept = *s_kept;
        __syncthreads();   // the block's LDS is rewritten next
    }
    for (int r = kept + tid; r < limit; r += kSelThreads) {
        a.keep[static_cast<int64_t>(c) * limit + r] = -1;
        a.kept_scores[static_cast<int64_t>(c) * limit + r] = 0.0f;
    }
    if (tid == 0) a.num_keep[c] = kept;
}

// Soft-NMS over the sorted candidates [base, base + n) of category c.  Candidates are
// dealt to threads (position r to thread r % 1024); up to kSoftReg per thread live in
// registers, the rest of a long category in global memory.
__device__ void select_soft(const NmsBatchArgs &a, int c, int base, int n, uint64_t *lds) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    uint64_t *wmin = lds;                                        // [2][kSelWaves]
    float4 *sbox = reinterpret_cast<float4 *>(lds + 2 * kSelWaves);   // [kSoftLdsBoxes]
    const bool lds_boxes = n <= kSoftLdsBoxes;
    if (lds_boxes)
        for (int r = tid; r < n; r += kSelThreads) sbox[r] = a.sbox[base + r];
    for (int r = kSoftReg * kSelThreads + tid; r < n; r += kSelThreads) a.skey[base + r] = 1;
    float s[kSoftReg];
    float4 bx[kSoftReg];
    uint32_t alive = 0;
#pragma unroll
    for (int m = 0; m < kSoftReg; ++m) {
        const int r = tid + m * kSelThreads;
        s[m] = 0.0f;
        bx[m] = make_float4(0, 0, 0, 0);
        if (r < n) {
            s[m] = a.sscore[base + r];
            bx[m] = a.sbox[base + r];
            alive |= 1u << m;
        }
    }
    __syncthreads();
    const int limit = a.max_keep;
    float4 last = make_float4(0, 0, 0, 0);
    bool have_last = false;
    int kept = 0;
    for (int it = 0; kept < limit; ++it) {
        // decay against the last selected box, drop, and this thread's best key
        uint64_t best = ~uint64_t(0);
#pragma unroll
        for (int m = 0; m < kSoftReg; ++m) {
            if (!((alive >> m) & 1)) continue;
            if (have_last) {
                s[m] = soft_decay(a, last, bx[m], s[m]);
                if (s[m] < a.score_threshold) {
                    alive &= ~(1u << m);
                    continue;
                }
            }
            const uint64_t key = (static_cast<uint64_t>(nms_key(s[m])) << 32) |
                                 static_cast<uint32_t>(tid + m * kSelThreads);
            best = key < best ? key : best;
        }
        // positions past the register slots keep their state in global memory: the
        // current score in sscore, alive in skey (free once the category is sorted)
        for (int r = tid + kSoftReg * kSelThreads; r < n; r += kSelThreads) {
            if (a.skey[base + r] == 0) continue;
            float sr = a.sscore[base + r];
            if (have_last) {
                sr = soft_decay(a, last, a.sbox[base + r], sr);
                a.sscore[base + r] = sr;
                if (sr < a.score_threshold) {
                    a.skey[base + r] = 0;
                    continue;
                }
            }
            const uint64_t key = (static_cast<uint64_t>(nms_key(sr)) << 32) | static_cast<uint32_t>(r);
            best = key < best ? key : best;
        }
        best = wave_min_u64(best);
        uint64_t *slot = wmin + (it & 1) * kSelWaves;
        if (lane == 0) slot[wave] = best;
        __syncthreads();
        uint64_t g = ~uint64_t(0);
#pragma unroll
        for (int w = 0; w < kSelWaves; ++w) g = slot[w] < g ? slot[w] : g;
        if (g == ~uint64_t(0)) break;   // uniform: no candidate left
        const int r = static_cast<int>(static_cast<uint32_t>(g));
        // the owner outputs the selected candidate with its current score and retires it
        if (r % kSelThreads == tid) {
            const int m = r / kSelThreads;
            float sc = 0.0f;
            if (m < kSoftReg) {
#pragma unroll
                for (int q = 0; q < kSoftReg; ++q)
                    if (q == m) sc = s[q];
                alive &= ~(1u << m);
            } else {
                sc = a.sscore[base + r];
                a.skey[base + r] = 0;
            }
            a.keep[static_cast<int64_t>(c) * limit + kept] = a.sidx[base + r];
            a.kept_scores[static_cast<int64_t>(c) * limit + kept] = sc;
        }
        ++kept;
        // every thread reads the selected box (its position is known to all)
        last = lds_boxes ? sbox[r] : a.sbox[base + r];
        have_last = true;
    }
    for (int q = kept + tid; q < limit; q += kSelThreads) {
        a.keep[static_cast<int64_t>(c) * limit + q] = -1;
        a.kept_scores[static_cast<int64_t>(c) * limit + q] = 0.0f;
    }
    if (tid == 0) a.num_keep[c] = kept;
}

__global__ __launch_bounds__(kSelThreads) void nmsb_select_kernel(NmsBatchArgs a) {
    __shared__ uint64_t lds[kSegLds];   // sort keys, then the selection's working set
    for (int c = blockIdx.x; c < a.C; c += gridDim.x) {
        const int base = a.start[c];
        const int n = a.start[c + 1] - base;
        // rank order: score rank key, then box index (unique keys)
        uint64_t *gkeys = a.skey + base;
        const bool in_lds = n <= kSegLds;
        for (int r = threadIdx.x; r < n; r += kSelThreads) {
            const int i = a.sidx[base + r];
            const uint64_t key = (static_cast<uint64_t>(nms_key(a.scores[i])) << 32) |
                                 static_cast<uint32_t>(i);
            if (in_lds) lds[r] = key;
            else gkeys[r] = key;
        }
        __syncthreads();
        if (in_lds) bitonic_sort_n(lds, n);
        else bitonic_sort_n(gkeys, n);
        for (int r = threadIdx.x; r < n; r += kSelThreads) {
            const uint64_t key = in_lds ? lds[r] : gkeys[r];
            const int i = static_cast<int>(static_cast<uint32_t>(key));
            a.sidx[base + r] = i;
            const float *bp = a.boxes + 4 * static_cast<int64_t>(i);
            a.sbox[base + r] = make_float4(bp[0], bp[1], bp[2], bp[3]);
            a.sscore[base + r] = a.scores[i];
        }
        __syncthreads();   // sorted arrays complete; the LDS is reused below
        if (a.method == kNmsHard) select_greedy(a, c, base, n, lds);
        else select_soft(a, c, base, n, lds);
        __syncthreads();   // before the next category reuses the LDS
    }
}

hipError_t launch_nms_batched(const NmsBatchArgs &a, hipStream_t stream) {
    nmsb_clear_kernel<<<std::max(1, std::min((a.C + 255) / 256, 256)), 256, 0, stream>>>(a.count,
                                                                                         a.C);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // contiguous ranges of kPlaceRange boxes, one workgroup each (N <= 2^24: at most 4096)
    const int blocks = static_cast<int>((static_cast<int64_t>(a.N) + kPlaceRange - 1) / kPlaceRange);
    const size_t hist_bytes = static_cast<size_t>(a.C) * sizeof(int32_t);
    if (a.N > 0) {
        nmsb_count_kernel<<<blocks, kPlaceThreads, hist_bytes, stream>>>(a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    const size_t shmem = static_cast<size_t>(a.C + kSelThreads) * sizeof(int32_t);
    nmsb_scan_kernel<<<1, kSelThreads, shmem, stream>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (a.N > 0) {
        nmsb_place_kernel<<<blocks, kPlaceThreads, hist_bytes, stream>>>(a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    nmsb_select_kernel<<<std::min(a.C, 4096), kSelThreads, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
