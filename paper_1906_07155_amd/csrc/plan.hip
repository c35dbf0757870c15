// plan.hip -- FPN level assignment and the RoI launch plan.
//
// Level assignment: §3.1 of MMDetection (SingleRoIExtractor pools each RoI from the
// FPN level matched to its size); the rule is the FPN rule in its threshold form,
// see include/roi_extract.h.
//
// The plan is a counting sort of the RoIs by (level, image, spatial cell of the box
// centre): RoIs that read the same feature rows end up next to each other in launch
// order, and the XCD-aware block mapping of the forward/backward then keeps them on
// one XCD's L2.  The order of RoIs with equal keys is whatever the atomics give;
// only the keys' order and the per-level offsets are defined.
//
// The plan also bins the RoIs into square bin-tiles of every (level, image) for
// the gather backward: a list of the RoIs whose footprint can reach each tile (a
// superset: a listed RoI may contribute nothing to the tile).
#include "internal.hpp"

namespace rex {

__global__ __launch_bounds__(256) void level_map_kernel(const float *__restrict__ rois,
                                                        int32_t K, int32_t L, float finest_scale,
                                                        int32_t box_plus1,
                                                        int32_t *__restrict__ out) {
    for (int32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x) {
        const float *r = rois + 5 * static_cast<int64_t>(k);
        out[k] = fpn_level(r[1], r[2], r[3], r[4], L, finest_scale, box_plus1);
    }
}

// Per-level values of the plan arguments, one 48-byte row per level staged in LDS
// at kernel start: a lane reads its level's row in one round trip (three 16-byte
// loads).  Indexing the argument arrays with a per-lane level would load from the
// argument segment per lane, and a select over the levels compiles to branches.
struct LevelRow {
    float scale;
    int32_t W, H, ncx, ncy, base, tbase, ntx, nty, dbase, band_base, band_rows;
};
struct LevelTab {
    LevelRow r[kMaxLevels];
};

// Threads 0..kMaxLevels-1 fill the table; a barrier must follow before it is read.
__device__ __forceinline__ void load_tab(const PlanArgs &a, LevelTab &t) {
    const int i = threadIdx.x;
    if (i < kMaxLevels) {
        LevelRow r;
        r.scale = a.scale[i];
        r.W = a.W[i];
        r.H = a.H[i];
        r.ncx = a.ncx[i];
        r.ncy = a.ncy[i];
        r.base = a.base[i];
        r.tbase = a.tbase[i];
        r.ntx = a.ntx[i];
        r.nty = a.nty[i];
        r.dbase = a.dbase[i];
        r.band_base = a.band_base[i];
        r.band_rows = a.band_rows[i];
        t.r[i] = r;
    }
}

__device__ __forceinline__ void roi_tile_box(const PlanArgs &a, const LevelRow &R, float x1,
                                             float y1, float x2, float y2, int &tx0, int &tx1,
                                             int &ty0, int &ty1) {
    roi_tile_range(x1, y1, x2, y2, R.scale, R.W, R.H, a.tile_shift, R.ntx, R.nty, tx0, tx1, ty0,
                   ty1);
}

// Sort key of a RoI: level bucket + image + spatial cell of the box centre.
__device__ __forceinline__ int plan_key(const PlanArgs &a, const LevelRow &R, float x1, float y1,
                                        float x2, float y2, int bb) {
    const int b = (bb < 0 || !a.batch_in_key) ? 0 : bb;
    float cx = (x1 + x2) * 0.5f * R.scale;
    float cy = (y1 + y2) * 0.5f * R.scale;
    cx = fminf(fmaxf(cx, 0.0f), static_cast<float>(R.W - 1));   // NaN -> 0
    cy = fminf(fmaxf(cy, 0.0f), static_cast<float>(R.H - 1));
    const int gx = min(static_cast<int>(cx) >> a.cell_shift, R.ncx - 1);
    const int gy = min(static_cast<int>(cy) >> a.cell_shift, R.ncy - 1);
    return R.base + (b * R.ncy + gy) * R.ncx + gx;
}

// Tile lists without a counting pass.  A list holds only RoIs of its own bucket
// (level l, image b), so the lists of that bucket fit in n_lb x T_l slots (n_lb RoIs
// in the bucket, T_l tiles per image on level l); the buckets take these regions in
// key order, which needs only the scanned key histogram, and sum to at most
// K x (the most tiles of one image-level) slots.  Each tile's list starts at
// tile_start[t] and ends at tile_end[t]; slots between lists stay unused.
//
// Tile t's bucket: level l, the first key of its (level, image) bucket, and its index
// inside the image's tiles (a function of the tile layout only).
struct TileBucket {
    int l, key0, local, T, ncell;
};

__device__ __forceinline__ TileBucket tile_bucket(const PlanArgs &a, int t) {
    int l = 0;
#pragma unroll
    for (int i = 1; i < kMaxLevels; ++i)
        if (i < a.L && t >= a.tbase[i]) l = i;
    // the level's values by a select chain over the (uniform) arguments
    int ntx = a.ntx[0], nty = a.nty[0], tbase = a.tbase[0], base = a.base[0];
    int ncell = a.ncx[0] * a.ncy[0];
#pragma unroll
    for (int i = 1; i < kMaxLevels; ++i) {
        const bool m = l == i;
        ntx = m ? a.ntx[i] : ntx;
        nty = m ? a.nty[i] : nty;
        tbase = m ? a.tbase[i] : tbase;
        base = m ? a.base[i] : base;
        ncell = m ? a.ncx[i] * a.ncy[i] : ncell;
    }
    const int T = ntx * nty;
    const int rel = t - tbase;
    // rel / T in binary32, exact (see box_row)
    const int b = static_cast<int>((static_cast<float>(rel) + 0.5f) *
                                   __builtin_amdgcn_rcpf(static_cast<float>(T)));
    return {l, base + b * ncell, rel - b * T, T, ncell};
}

// Start of the list of a tile of bucket x; bstart(key) is the first plan slot of `key`
// (K for nbins).
template <typename F>
__device__ __forceinline__ int tile_region(const PlanArgs &a, const TileBucket &x, F &&bstart) {
    // first slots of the levels (uniform addresses, loaded together), and the slots
    // of the levels before l: each RoI of level i with T_i tiles
    int ls[kMaxLevels];
#pragma unroll
    for (int i = 0; i < kMaxLevels; ++i) ls[i] = i < a.L ? bstart(a.base[i]) : a.K;
    const int bs = bstart(x.key0);
    const int be = bstart(x.key0 + x.ncell);
    int r = 0, lo = ls[0];
#pragma unroll
    for (int i = 0; i < kMaxLevels - 1; ++i) {
        if (i < x.l) {
            r += (ls[i + 1] - ls[i]) * a.ntx[i] * a.nty[i];
            lo = ls[i + 1];
        }
    }
    return r + (bs - lo) * x.T + x.local * (be - bs);
}

// Row of tile i (row-major) of a w-wide box: (i + 1/2) / w in binary32 with the
// hardware reciprocal (1 ulp), exact for 0 <= i < 2^21 - 1: the relative error of the
// reciprocal and the product, below 2^-22, leaves (i + 1/2) / w within (i + 1/2) 2^-22
// / w < 1 / (2w) of its value, less than its distance to the nearest integer.  Tile
// counts here are at most kPlanMaxBins.
__device__ __forceinline__ int box_row(int i, float rw) {
    return static_cast<int>((static_cast<float>(i) + 0.5f) * rw);
}

// The tile phases of the multi-kernel plan give each RoI kPlanLanes consecutive lanes,
// which split its tiles, so the atomics of one RoI are in flight together.
constexpr int kPlanLanes = 16;

// ---------------------------------------------------------------------------
// One-launch plan (up to kPlanOne RoIs): one 1024-thread workgroup per role, none
// waiting for another.
//   block 0: the sort -- levels, keys, the LDS key histogram and its scan, per-level
//            offsets, the permutation;
//   block 1: the tile order -- every tile's list length from a difference grid (four
//            LDS atomics per RoI at the corners of its tile box, then prefix sums along
//            x and along y), and the longest-first counting sort;
//   blocks 2..: one band of tile rows of one (level, image) each -- the bucket sizes
//            that place its lists (wave ballots over all RoIs), then the lists of its
//            own tiles.
// A single workgroup issues 64 lanes per cycle; splitting the list fill over the
// bands keeps every role to a few instructions per RoI.
// ---------------------------------------------------------------------------
constexpr int kPlanOne = 8192;

constexpr int kPlanWords = 24576;  // 96 KiB of LDS per workgroup

// fn(k, roi) for every RoI, each thread's RoIs loaded kRoiBatch at a time.
template <typename F>
__device__ __forceinline__ void for_rois(const PlanArgs &a, F &&fn) {
    constexpr int kRoiBatch = 4;
    for (int base = 0; base < a.K; base += kRoiBatch * kPlanThreads) {
        float rv[kRoiBatch][5];
#pragma unroll
        for (int i = 0; i < kRoiBatch; ++i) {
            const int k = base + static_cast<int>(threadIdx.x) + i * kPlanThreads;
            if (k < a.K) {
                const float *r = a.rois + 5 * static_cast<int64_t>(k);
#pragma unroll
                for (int j = 0; j < 5; ++j) rv[i][j] = r[j];
            }
        }
#pragma unroll
        for (int i = 0; i < kRoiBatch; ++i) {
            const int k = base + static_cast<int>(threadIdx.x) + i * kPlanThreads;
            if (k < a.K) fn(k, rv[i]);
        }
    }
}

// Exact quotient of non-negative integers n < 2^21 - 1 and d >= 1.
__device__ __forceinline__ int small_div(int n, int d) { return small_div_exact(n, d); }

__device__ void plan_sort_role(const PlanArgs &a, const LevelTab &tb, int32_t *smem) {
    int32_t *hist = smem;                  // [nbins]
    int32_t *part = hist + a.nbins;        // [kPlanThreads]
    int32_t *keys = part + kPlanThreads;   // [K]
    const int tid = threadIdx.x;
    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = 0;
    __syncthreads();
    // a1: the level of every RoI and its key (level bucket + image + spatial cell)
    for_rois(a, [&](int k, const float (&r)[5]) {
        const int lvl = fpn_level(r[1], r[2], r[3], r[4], a.L, a.finest_scale, a.box_plus1);
        a.levels_out[k] = lvl;
        const int key = plan_key(a, tb.r[lvl], r[1], r[2], r[3], r[4], roi_batch(r[0], a.N));
        keys[k] = key;
        atomicAdd(&hist[key], 1);
    });
    __syncthreads();
    block_exclusive_scan(hist, a.nbins, part);
    if (tid == 0) {
#pragma unroll
        for (int l = 0; l < kMaxLevels; ++l)
            if (l < a.L) a.offsets[l] = hist[tb.r[l].base];
        a.offsets[a.L] = a.K;
    }
    __syncthreads();   // the offsets are read before the cursors move
    // a2: every RoI index to its slot (hist becomes the bucket cursors)
    for (int k = tid; k < a.K; k += kPlanThreads) {
        const int pos = atomicAdd(&hist[keys[k]], 1);
        if (pos < a.K) a.perm[pos] = k;
    }
}

__device__ void plan_order_role(const PlanArgs &a, const LevelTab &tb, int32_t *smem) {
    int32_t *diff = smem;                  // [ndiff]: per tile row, +1 / -1 at a box's ends
    int32_t *lens = diff + a.ndiff;        // [ntiles]: list lengths
    int32_t *part = lens + a.ntiles;       // [kPlanThreads]
    constexpr int kLenBins = 256;
    int32_t *lenh = part + 2 * (kPlanThreads / 64) + 1;   // after the scan scratch
    const int tid = threadIdx.x;
    for (int i = tid; i < a.ndiff; i += kPlanThreads) diff[i] = 0;
    if (tid < kLenBins) lenh[tid] = 0;
    __syncthreads();
    // every tile row a RoI's box meets: +1 at its first tile, -1 past its last
    for_rois(a, [&](int, const float (&r)[5]) {
        const int bb = roi_batch(r[0], a.N);
        if (bb < 0) return;
        const LevelRow R =
            tb.r[fpn_level(r[1], r[2], r[3], r[4], a.L, a.finest_scale, a.box_plus1)];
        int tx0, tx1, ty0, ty1;
        roi_tile_box(a, R, r[1], r[2], r[3], r[4], tx0, tx1, ty0, ty1);
        const int W1 = R.ntx + 1;
        int d = R.dbase + (bb * (R.nty + 1) + ty0) * W1;
        for (int y = ty0; y <= ty1; ++y, d += W1) {
            atomicAdd(&diff[d + tx0], 1);
            atomicAdd(&diff[d + tx1 + 1], -1);
        }
    });
    __syncthreads();
    // prefix sums along each tile row (one row per thread, kRun values per round
    // trip): the list lengths, binned by length on the way
    int nrows = 0;
#pragma unroll
    for (int l = 0; l < kMaxLevels; ++l)
        if (l < a.L) nrows += a.N * tb.r[l].nty;
    constexpr int kRun = 32;
    for (int i = tid; i < nrows; i += kPlanThreads) {
        int l = 0, first = 0, acc = 0;
#pragma unroll
        for (int j = 0; j < kMaxLevels; ++j)
            if (j < a.L) {
                if (i >= acc) {
                    l = j;
                    first = acc;
                }
                acc += a.N * tb.r[j].nty;
            }
        const LevelRow &R = tb.r[l];
        const int row = i - first;                 // image * nty + y
        const int b = small_div(row, R.nty);
        const int base = R.dbase + (row + b) * (R.ntx + 1);   // (b (nty + 1) + y) (ntx + 1)
        const int t0 = R.tbase + row * R.ntx;
        int run = 0;
        for (int x0 = 0; x0 < R.ntx; x0 += kRun) {
            int v[kRun];
#pragma unroll
            for (int u = 0; u < kRun; ++u) v[u] = x0 + u < R.ntx ? diff[base + x0 + u] : 0;
#pragma unroll
            for (int u = 0; u < kRun; ++u) {
                run += v[u];
                if (x0 + u < R.ntx) {
                    const int len = min(max(run, 0), kLenBins - 1);
                    lens[t0 + x0 + u] = len;
                    atomicAdd(&lenh[kLenBins - 1 - len], 1);
                }
            }
        }
    }
    __syncthreads();
    block_exclusive_scan(lenh, kLenBins, part);
    for (int t = tid; t < a.ntiles; t += kPlanThreads) {
        const int pos = atomicAdd(&lenh[kLenBins - 1 - lens[t]], 1);
        if (pos >= 0 && pos < a.ntiles) a.tile_order[pos] = t;
    }
}

__device__ void plan_band_role(const PlanArgs &a, const LevelTab &tb, int32_t *smem, int band) {
    int32_t *cur = smem;                        // [kBandTiles]: next free slot per tile
    int32_t *cand = cur + kBandTiles;           // [3 * kBandCand]: RoI, x range, y range
    int32_t *pre = cand + 3 * kBandCand;        // [kBandCand]: first pair of each kept RoI
    int32_t *part = pre + kBandCand;            // [kPlanThreads]: scan scratch
    int32_t *cnt = part + kPlanThreads;         // [kMaxLevels + 3]
    const int tid = threadIdx.x;
    if (tid < kMaxLevels + 3) cnt[tid] = 0;
    __syncthreads();   // the level table is read only after this barrier
    // the band: rows [ty0, ty1) of image b on level l (uniform)
    int l = 0;
#pragma unroll
    for (int i = 1; i < kMaxLevels; ++i)
        if (i < a.L && band >= tb.r[i].band_base) l = i;
    const LevelRow &R = tb.r[l];
    const int per_img = (R.nty + R.band_rows - 1) / R.band_rows;
    const int j = band - R.band_base;
    const int b = j / per_img;
    const int ty0 = (j - b * per_img) * R.band_rows;
    const int ty1 = min(ty0 + R.band_rows, R.nty);
    const int nbt = (ty1 - ty0) * R.ntx;
    const int tile0 = R.tbase + (b * R.nty + ty0) * R.ntx;

    // Bucket sizes: RoIs per level, and on level l those of images before b and of
    // image b (an invalid image counts as image 0, as in the keys).  RoIs of (l, b)
    // whose tile rows meet the band are kept.
    int lc[kMaxLevels];
#pragma unroll
    for (int i = 0; i < kMaxLevels; ++i) lc[i] = 0;
    int before = 0, inb = 0;
    auto keep = [&](int k, const float (&r)[5]) {
        int tx0, tx1, ry0, ry1;
        roi_tile_box(a, R, r[1], r[2], r[3], r[4], tx0, tx1, ry0, ry1);
        if (ry1 < ty0 || ry0 >= ty1) return;
        const int c = atomicAdd(&cnt[kMaxLevels + 2], 1);
        if (c < kBandCand) {
            cand[3 * c] = k;
            cand[3 * c + 1] = tx0 | (tx1 << 16);
            cand[3 * c + 2] = max(ry0, ty0) | (min(ry1, ty1 - 1) << 16);
        }
    };
    for_rois(a, [&](int k, const float (&r)[5]) {
        const int lvl = fpn_level(r[1], r[2], r[3], r[4], a.L, a.finest_scale, a.box_plus1);
        const int bb = roi_batch(r[0], a.N);
        const int bk = bb < 0 ? 0 : bb;
#pragma unroll
        for (int i = 0; i < kMaxLevels; ++i)
            if (i < a.L) lc[i] += __popcll(__ballot(lvl == i));
        before += __popcll(__ballot(lvl == l && bk < b));
        inb += __popcll(__ballot(lvl == l && bk == b));
        if (lvl == l && bb == b) keep(k, r);
    });
    if ((tid & 63) == 0) {
#pragma unroll
        for (int i = 0; i < kMaxLevels; ++i)
            if (i < a.L) atomicAdd(&cnt[i], lc[i]);
        atomicAdd(&cnt[kMaxLevels], before);
        atomicAdd(&cnt[kMaxLevels + 1], inb);
    }
    __syncthreads();

    // The lists of bucket (l, b) start after those of the RoIs of earlier levels (T_i
    // slots each) and of earlier images on level l (T_l slots each); a tile's list has
    // room for every RoI of the bucket.
    int first = 0;
#pragma unroll
    for (int i = 0; i < kMaxLevels; ++i)
        if (i < l) first += cnt[i] * tb.r[i].ntx * tb.r[i].nty;
    const int n = cnt[kMaxLevels + 1];
    first += cnt[kMaxLevels] * R.ntx * R.nty + ty0 * R.ntx * n;   // tile (ty0, 0)
    for (int i = tid; i < nbt; i += kPlanThreads) cur[i] = first + i * n;
    __syncthreads();

    auto fill = [&](int k, int x0, int x1, int y0, int y1) {
        for (int y = y0; y <= y1; ++y)
            for (int x = x0; x <= x1; ++x) {
                const int p = atomicAdd(&cur[(y - ty0) * R.ntx + x], 1);
                if (p < a.capacity) a.tile_rois[p] = k;
            }
    };
    const int nc = cnt[kMaxLevels + 2];
    if (nc <= kBandCand) {
        // one (RoI, tile) pair per lane: the kept RoIs' tile counts in the band, their
        // prefix sums, and for pair p the RoI whose range holds it (binary search)
        for (int c = tid; c < nc; c += kPlanThreads) {
            const int xr = cand[3 * c + 1], yr = cand[3 * c + 2];
            pre[c] = ((xr >> 16) - (xr & 0xffff) + 1) * ((yr >> 16) - (yr & 0xffff) + 1);
        }
        __syncthreads();
        const int pairs = block_exclusive_scan(pre, nc, part);
        for (int p = tid; p < pairs; p += kPlanThreads) {
            int lo = 0, hi = nc - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (pre[mid] <= p) lo = mid;
                else hi = mid - 1;
            }
            const int xr = cand[3 * lo + 1], yr = cand[3 * lo + 2];
            const int x0 = xr & 0xffff, w = (xr >> 16) - x0 + 1;
            const int i = p - pre[lo];
            const int dy = small_div(i, w);
            const int y = (yr & 0xffff) + dy;
            const int q = atomicAdd(&cur[(y - ty0) * R.ntx + x0 + (i - dy * w)], 1);
            if (q < a.capacity) a.tile_rois[q] = cand[3 * lo];
        }
    } else {
        for_rois(a, [&](int k, const float (&r)[5]) {
            if (roi_batch(r[0], a.N) != b ||
                fpn_level(r[1], r[2], r[3], r[4], a.L, a.finest_scale, a.box_plus1) != l)
                return;
            int tx0, tx1, ry0, ry1;
            roi_tile_box(a, R, r[1], r[2], r[3], r[4], tx0, tx1, ry0, ry1);
            if (ry1 < ty0 || ry0 >= ty1) return;
            fill(k, tx0, tx1, max(ry0, ty0), min(ry1, ty1 - 1));
        });
    }
    __syncthreads();
    for (int i = tid; i < nbt; i += kPlanThreads) {
        a.tile_start[tile0 + i] = first + i * n;
        a.tile_end[tile0 + i] = cur[i];
    }
}

__global__ __launch_bounds__(kPlanThreads) void plan_one_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    __shared__ LevelTab tb;
    load_tab(a, tb);   // every role reads the table only after its first barrier
    if (blockIdx.x == 0)
        plan_sort_role(a, tb, smem);
    else if (blockIdx.x == 1)
        plan_order_role(a, tb, smem);
    else
        plan_band_role(a, tb, smem, static_cast<int>(blockIdx.x) - 2);
}

// LDS words of the one-launch plan's roles, and whether it takes these arguments.
__host__ __device__ inline int plan_one_words(const PlanArgs &a) {
    int w = a.nbins + kPlanThreads + a.K;
    if (a.ntiles > 0) {
        w = max(w, a.ndiff + a.ntiles + kPlanThreads);
        w = max(w, kBandTiles + 4 * kBandCand + kPlanThreads + kMaxLevels + 3);
    }
    return w;
}

// Larger plans run as five short kernels over the whole GPU: clear the key counters;
// per RoI, its level and sort key, counted with device-scope integer atomics; one
// workgroup turns the counts into bucket starts, per-level offsets and the first slot
// of every tile list; per RoI, its slot in the permutation and in each of its tiles'
// lists; one workgroup orders the tiles by list length.

__global__ __launch_bounds__(256) void plan_clear_kernel(int32_t *__restrict__ a, int32_t na) {
    for (int32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < na; i += gridDim.x * blockDim.x)
        a[i] = 0;
}

__global__ __launch_bounds__(256) void plan_count_kernel(PlanArgs a) {
    __shared__ LevelTab tb;
    load_tab(a, tb);
    __syncthreads();
    for (int64_t k = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; k < a.K;
         k += static_cast<int64_t>(gridDim.x) * 256) {
        const float *r = a.rois + 5 * k;
        const float b0 = r[0], x1 = r[1], y1 = r[2], x2 = r[3], y2 = r[4];
        const int lvl = fpn_level(x1, y1, x2, y2, a.L, a.finest_scale, a.box_plus1);
        const int bb = roi_batch(b0, a.N);
        a.levels_out[k] = lvl;
        const int key = plan_key(a, tb.r[lvl], x1, y1, x2, y2, bb);
        a.keys[k] = key;
        atomicAdd(&a.key_count[key], 1);
    }
}

__global__ __launch_bounds__(kPlanThreads) void plan_scan_kernel(PlanArgs a) {
    extern __shared__ int32_t smem[];
    int32_t *hist = smem;                    // [nbins]
    int32_t *part = smem + a.nbins;          // [kPlanThreads]
    const int tid = threadIdx.x;

    // Bucket starts (the fill kernel's cursors), per-level offsets, list starts.
    for (int i = tid; i < a.nbins; i += kPlanThreads) hist[i] = a.key_count[i];
    __syncthreads();
    block_exclusive_scan(hist, a.nbins, part);
    for (int i = tid; i < a.nbins; i += kPlanThreads) a.key_count[i] = hist[i];
    if (tid == 0) {
#pragma unroll
        for (int l = 0; l < kMaxLevels; ++l)
            if (l < a.L) a.offsets[l] = hist[a.base[l]];
        a.offsets[a.L] = a.K;
    }
    const int nb = a.nbins, K = a.K;
    auto bstart = [&](int key) { return key < nb ? hist[key] : K; };
    for (int t = tid; t < a.ntiles; t += kPlanThreads) {
        const int r = tile_region(a, tile_bucket(a, t), bstart);
        a.tile_start[t] = r;
        a.tile_end[t] = r;   // the fill kernel's cursor
    }
}

__global__ __launch_bounds__(256) void plan_fill_kernel(PlanArgs a) {
    __shared__ LevelTab tb;
    load_tab(a, tb);
    __syncthreads();
    const int sub = threadIdx.x % kPlanLanes;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * (256 / kPlanLanes);
    for (int64_t k = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) / kPlanLanes; k < a.K;
         k += stride) {
        if (sub == 0) {
            const int pos = atomicAdd(&a.key_count[a.keys[k]], 1);
            if (pos < a.K) a.perm[pos] = static_cast<int32_t>(k);
        }
        if (a.ntiles > 0) {
            const float *r = a.rois + 5 * k;
            const int bb = roi_batch(r[0], a.N);
            if (bb < 0) continue;
            const int lvl = a.levels_out[k];
            int tx0, tx1, ty0, ty1;
            const LevelRow R = tb.r[lvl];
            roi_tile_box(a, R, r[1], r[2], r[3], r[4], tx0, tx1, ty0, ty1);
            const int w = tx1 - tx0 + 1;
            const int n = w * (ty1 - ty0 + 1);
            const float rw = __builtin_amdgcn_rcpf(static_cast<float>(w));
            const int ntx = R.ntx;
            const int base = R.tbase + bb * R.nty * ntx;
            for (int i = sub; i < n; i += kPlanLanes) {
                const int dy = box_row(i, rw);
                const int t = base + (ty0 + dy) * ntx + tx0 + (i - dy * w);
                const int p = atomicAdd(&a.tile_end[t], 1);
                if (p < a.capacity) a.tile_rois[p] = static_cast<int32_t>(k);
            }
        }
    }
}

__global__ __launch_bounds__(kPlanThreads) void plan_order_kernel(PlanArgs a) {
    __shared__ int32_t part[kPlanThreads];
    constexpr int kLenBins = 256;
    int32_t *lenh = part + 2 * (kPlanThreads / 64) + 1;   // after the scan scratch
    const int tid = threadIdx.x;
    if (tid < kLenBins) lenh[tid] = 0;
    __syncthreads();
    for (int t = tid; t < a.ntiles; t += kPlanThreads)
        atomicAdd(&lenh[kLenBins - 1 - min(a.tile_end[t] - a.tile_start[t], kLenBins - 1)], 1);
    __syncthreads();
    block_exclusive_scan(lenh, kLenBins, part);
    for (int t = tid; t < a.ntiles; t += kPlanThreads) {
        const int len = a.tile_end[t] - a.tile_start[t];
        const int pos = atomicAdd(&lenh[kLenBins - 1 - min(len, kLenBins - 1)], 1);
        a.tile_order[pos] = t;
    }
}

hipError_t launch_level_map(const float *rois, int32_t K, int32_t L, float finest_scale,
                            int32_t box_plus1, int32_t *out, hipStream_t stream) {
    const int blocks = min((K + 255) / 256, 4096);
    level_map_kernel<<<blocks, 256, 0, stream>>>(rois, K, L, finest_scale, box_plus1, out);
    return hipGetLastError();
}

hipError_t launch_plan(const PlanArgs &a, hipStream_t stream) {
    const int words = plan_one_words(a);
    if (a.K <= kPlanOne && words <= kPlanWords && (a.ntiles <= 0 || a.nbands > 0)) {
        const int grid = a.ntiles > 0 ? 2 + a.nbands : 1;
        plan_one_kernel<<<grid, kPlanThreads, static_cast<size_t>(words) * sizeof(int32_t),
                          stream>>>(a);
        return hipGetLastError();
    }
    plan_clear_kernel<<<max(1, min((a.nbins + 255) / 256, 1024)), 256, 0, stream>>>(a.key_count,
                                                                                a.nbins);
    plan_count_kernel<<<max(1, min((a.K + 255) / 256, 4096)), 256, 0, stream>>>(a);
    const size_t shmem = static_cast<size_t>(a.nbins + kPlanThreads) * sizeof(int32_t);
    plan_scan_kernel<<<1, kPlanThreads, shmem, stream>>>(a);
    const int blocks = max(1, min((a.K + 256 / kPlanLanes - 1) / (256 / kPlanLanes), 4096));
    plan_fill_kernel<<<blocks, 256, 0, stream>>>(a);
    if (a.ntiles > 0) plan_order_kernel<<<1, kPlanThreads, 0, stream>>>(a);
    return hipGetLastError();
}

}  // namespace rex
