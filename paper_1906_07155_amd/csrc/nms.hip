// nms.hip -- greedy non-maximum suppression of scored boxes.
//
// The proposals a two-stage detector extracts RoI features for come out of NMS over
// the dense head's scored boxes; MMDetection runs such bbox operations on the GPU (§1).
// Definition (rank order, tie rules, binary32 IoU decision) in include/roi_extract.h.
//
// Three kernels on one stream:
//   nms_sort_kernel   one 1024-thread workgroup: every box becomes a 64-bit item
//                     (rank key << 32 | index), and a bitonic network in LDS sorts them
//                     (key first, index second); the boxes and categories are then
//                     gathered in rank order.
//   nms_mask_kernel   one 64-lane workgroup per (row block, column block) of the upper
//                     triangle: lane r of row block I tests its box against the 64 boxes
//                     of column block J (staged in LDS) and writes the 64-bit mask of
//                     later boxes of its category that it overlaps by IoU > threshold.
//   nms_scan_kernel   one 1024-thread workgroup walks the row blocks in rank order: wave
//                     0 resolves a block sequentially from its diagonal masks (one lane
//                     read per box) and writes the kept indices; then every thread ORs the
//                     kept rows of its group into its later words and adds them to the
//                     removal words in LDS (lanes over words, so an atomic instruction
//                     touches 64 different words), the rows having been loaded three
//                     blocks ahead so their latency hides behind the resolution.
#include "internal.hpp"

namespace rex {

constexpr int kNmsSortThreads = 1024;

__global__ __launch_bounds__(kNmsSortThreads) void nms_sort_kernel(NmsArgs a) {
    __shared__ uint64_t items[kNmsMaxBoxes];
    const int N = a.N;
    int P = 1;
    while (P < N) P <<= 1;
    for (int i = threadIdx.x; i < P; i += kNmsSortThreads) {
        uint64_t v = (static_cast<uint64_t>(0xffffffffu) << 32) | 0x7fffffffu;   // pad: last
        if (i < N) v = (static_cast<uint64_t>(nms_key(a.scores[i])) << 32) | static_cast<uint32_t>(i);
        items[i] = v;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            // the P / 2 compare-exchange pairs (i, i + j), i with bit j clear
            for (int q = threadIdx.x; q < P / 2; q += kNmsSortThreads) {
                const int i = ((q & ~(j - 1)) << 1) | (q & (j - 1));
                const int p = i + j;
                const uint64_t x = items[i], y = items[p];
                const bool up = (i & k) == 0;
                if ((x > y) == up) {
                    items[i] = y;
                    items[p] = x;
                }
            }
            // With j <= 64 the 64 pairs of a wave (64 consecutive q) cover one aligned
            // block of 128 items, the same block for every such j: between two such
            // stages each wave only reads what it wrote, so a wave-level sync suffices.
            // Any stage with partners 128 or more apart, and the end of the sort (the
            // gather below reads every item), needs the workgroup barrier.
            const int jn = j > 1 ? j >> 1 : k;   // next stage's distance
            if (j <= 64 && jn <= 64 && !(k == P && j == 1))
                wave_sync();
            else
                __syncthreads();
        }
    }
    for (int r = threadIdx.x; r < N; r += kNmsSortThreads) {
        const int idx = static_cast<int>(static_cast<uint32_t>(items[r]));
        a.order[r] = idx;
        const float *b = a.boxes + 4 * static_cast<int64_t>(idx);
        a.sboxes[r] = make_float4(b[0], b[1], b[2], b[3]);
        a.scats[r] = a.categories ? a.categories[idx] : 0;
    }
}

__global__ __launch_bounds__(64) void nms_mask_kernel(NmsArgs a) {
    __shared__ float4 sb[64];
    __shared__ int sc[64];
    const int nb = a.nw;
    const int ib = static_cast<int>(blockIdx.x) / nb;
    const int jb = static_cast<int>(blockIdx.x) - ib * nb;
    if (jb < ib) return;   // uniform over the workgroup: the lower triangle is never read
    const int lane = threadIdx.x;
    const int j0 = jb * 64;
    if (j0 + lane < a.N) {
        sb[lane] = a.sboxes[j0 + lane];
        sc[lane] = a.scats[j0 + lane];
    }
    __syncthreads();
    const int i = ib * 64 + lane;
    if (i >= a.N) return;
    const float4 bi = a.sboxes[i];
    const int ci = a.scats[i];
    const int jn = min(64, a.N - j0);
    uint64_t bits = 0;
    for (int jj = 0; jj < jn; ++jj) {
        const int j = j0 + jj;
        if (j > i && sc[jj] == ci && nms_iou(bi, sb[jj]) > a.threshold) bits |= uint64_t(1) << jj;
    }
    a.mask[static_cast<int64_t>(i) * nb + jb] = bits;
}

// A block's propagation over the scan workgroup: waves over groups of rows, lanes over
// later words.
constexpr int kNmsScanThreads = 1024;
constexpr int kNmsRowsPerWave = 64 / (kNmsScanThreads / 64);           // 4
constexpr int kNmsWordsPerLane = (kNmsMaxBoxes / 64 + 63) / 64;        // 2
constexpr int kNmsPairs = kNmsRowsPerWave * kNmsWordsPerLane;
constexpr int kNmsAhead = 3;   // blocks of mask rows in flight ahead of the one resolved

__global__ __launch_bounds__(kNmsScanThreads) void nms_scan_kernel(NmsArgs a) {
    __shared__ uint64_t removed[kNmsMaxBoxes / 64];
    __shared__ uint64_t s_keptm[kNmsMaxBoxes / 64];   // kept boxes of every resolved block
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int nb = a.nw;
    const int limit = static_cast<int>(min<int64_t>(a.max_keep, a.N));
    for (int w = tid; w < nb; w += kNmsScanThreads) removed[w] = 0;

    // Rows of a block as loaded ahead: wave 0 its diagonal words, every thread its share
    // of the (row, later word) pairs.
    auto load_diag = [&](int b) -> uint64_t {
        const int i = b * 64 + lane;
        return (b < nb && i < a.N) ? a.mask[static_cast<int64_t>(i) * nb + b] : 0;
    };
    // thread (wave, lane) holds rows 4 wave .. 4 wave + 3 of the block at the later words
    // b + 1 + lane and b + 65 + lane: pf[4 j + r] = row 4 wave + r, word b + 1 + lane + 64 j
    auto load_pairs = [&](int b, uint64_t (&pf)[kNmsPairs]) {
#pragma unroll
        for (int j = 0; j < kNmsWordsPerLane; ++j) {
#pragma unroll
            for (int r = 0; r < kNmsRowsPerWave; ++r) {
                const int w = b + 1 + lane + 64 * j;
                const int row = b * 64 + wave * kNmsRowsPerWave + r;
                pf[j * kNmsRowsPerWave + r] =
                    (b < nb && w < nb && row < a.N) ? a.mask[static_cast<int64_t>(row) * nb + w] : 0;
            }
        }
    };
    // Rows of the next kNmsAhead blocks are in flight: slot 0 holds block b, the loads
    // of block b + kNmsAhead are issued as block b starts.
    uint64_t pf[kNmsAhead][kNmsPairs];
    uint64_t dg[kNmsAhead];
#pragma unroll
    for (int d = 0; d < kNmsAhead; ++d) {
        dg[d] = wave == 0 ? load_diag(d) : 0;
        load_pairs(d, pf[d]);
    }
    __syncthreads();
    int count = 0;   // the same in every thread
    int nres = 0;    // blocks resolved
    for (int b = 0; b < nb; ++b) {
        const uint64_t dg_new = wave == 0 ? load_diag(b + kNmsAhead) : 0;
        uint64_t pf_new[kNmsPairs];
        load_pairs(b + kNmsAhead, pf_new);
        if (wave == 0) {
            // sequential within the block: box t is kept unless a kept box of an earlier
            // block or an earlier kept box of this block removed it.  The removal word is
            // the same in every lane; held in scalar registers, each step is a scalar
            // branch instead of a masked vector one.
            const int nrow = min(64, a.N - b * 64);
            const uint64_t rw = removed[b];
            // (readfirstlane returns a signed int: both halves go through uint32_t, so
            // the low half is not sign-extended into the high one)
            const uint32_t rlo = static_cast<uint32_t>(
                __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(rw)));
            const uint32_t rhi = static_cast<uint32_t>(
                __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(rw >> 32)));
            uint64_t rem = (static_cast<uint64_t>(rhi) << 32) | rlo;
            uint64_t kept = 0;
            for (int t = 0; t < nrow; ++t) {
                if (!((rem >> t) & 1)) {
                    kept |= uint64_t(1) << t;
                    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<uint32_t>(dg[0]), t);
                    const uint32_t hi =
                        __builtin_amdgcn_readlane(static_cast<uint32_t>(dg[0] >> 32), t);
                    rem |= (static_cast<uint64_t>(hi) << 32) | lo;
                }
            }
            if (lane == 0) s_keptm[b] = kept;   // indices are written after the loop
        }
        __syncthreads();
        const uint64_t kept = s_keptm[b];
        count += __popcll(kept);
        nres = b + 1;
        if (count >= limit) break;   // uniform over the workgroup
        // the kept rows remove boxes of later blocks: each thread ORs its kept rows of a
        // word, then adds them to the word in LDS (the 64 lanes of an atomic instruction
        // address 64 different words)
#pragma unroll
        for (int j = 0; j < kNmsWordsPerLane; ++j) {
            uint64_t v = 0;
#pragma unroll
            for (int r = 0; r < kNmsRowsPerWave; ++r)
                if ((kept >> (wave * kNmsRowsPerWave + r)) & 1) v |= pf[0][j * kNmsRowsPerWave + r];
            const int w = b + 1 + lane + 64 * j;
            if (v != 0 && w < nb)
                atomicOr(reinterpret_cast<unsigned long long *>(&removed[w]),
                         static_cast<unsigned long long>(v));
        }
#pragma unroll
        for (int d = 0; d + 1 < kNmsAhead; ++d) {
            dg[d] = dg[d + 1];
#pragma unroll
            for (int m = 0; m < kNmsPairs; ++m) pf[d][m] = pf[d + 1][m];
        }
        dg[kNmsAhead - 1] = dg_new;
#pragma unroll
        for (int m = 0; m < kNmsPairs; ++m) pf[kNmsAhead - 1][m] = pf_new[m];
        __syncthreads();   // removal words final before block b + 1 is resolved
    }
    // Kept indices in rank order, off the sequential path: wave w writes blocks w,
    // w + 16, ...; a block's first rank is the kept count of the blocks before it.
    __syncthreads();
    for (int b = wave; b < nres; b += kNmsScanThreads / 64) {
        int before = 0;
        for (int c = lane; c < b; c += 64) before += __popcll(s_keptm[c]);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) before += __shfl_xor(before, o, 64);
        const uint64_t kept = s_keptm[b];
        if ((kept >> lane) & 1) {
            const int rank = before + __popcll(kept & ((uint64_t(1) << lane) - 1));
            if (rank < limit) a.keep[rank] = a.order[b * 64 + lane];
        }
    }
    const int n = min(count, limit);
    for (int r = n + tid; r < limit; r += kNmsScanThreads) a.keep[r] = -1;
    if (tid == 0) a.num_keep[0] = n;
}

hipError_t launch_nms(NmsArgs a, hipStream_t stream) {
    if (a.N == 0) {
        // nothing kept: the count is written by the scan with an empty loop
        nms_scan_kernel<<<1, kNmsScanThreads, 0, stream>>>(a);
        return hipGetLastError();
    }
    nms_sort_kernel<<<1, kNmsSortThreads, 0, stream>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    nms_mask_kernel<<<static_cast<uint32_t>(a.nw * a.nw), 64, 0, stream>>>(a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    nms_scan_kernel<<<1, kNmsScanThreads, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
