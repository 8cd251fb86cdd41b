// Depth-sorted per-tile lists (Sec. 3.1 "depth-sorted order"): the pairs must
// come out ordered by (tile, depth key, Gaussian index).
//
// Instead of radix-sorting P 45-bit (tile, depth) keys, the Gaussians are
// sorted once by depth (4 stable 8-bit LSD passes over n 32-bit keys with the
// index as value, so equal depths stay in index order), the pairs are emitted
// in that order, and a stable LSD sort on the tile id alone finishes the job:
// stability keeps (depth, index) order within a tile. The tile id needs
// ceil(log2 T) bits, split evenly over as few passes of <= 8 bits as possible.
//
// One radix pass = k_radix_hist (per-workgroup digit counts) + k_radix_scan
// (exclusive offsets per digit over workgroups) + k_radix_scatter: each wave
// ranks a contiguous slice of the workgroup's keys with ballot-matched digits
// (no workgroup barrier per round), the workgroup reorders its keys (4096 in
// the depth sort, 6144 in the tile sort) by digit in LDS, and writes each
// digit's run to consecutive global addresses.
#include "gs_internal.h"

namespace gsr {

namespace {

constexpr int kDupItems = kDupChunk / kBlock;              // 4 per thread

__device__ __forceinline__ uint64_t lanemask_lt() { return (1ull << __lane_id()) - 1ull; }

// Exclusive scan of one u32 per thread over the 256-thread workgroup.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* lds4, uint32_t* total)
{
    const int lane = __lane_id(), wave = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) lds4[wave] = x;
    __syncthreads();
    uint32_t before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const uint32_t s = lds4[w];
        if (w < wave) before += s;
        tot += s;
    }
    __syncthreads();
    if (total) *total = tot;
    return before + x - v;
}

// Lanes of this wave holding the same kBits-bit digit (restricted to valid lanes).
template <int kBits>
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid)
{
    const uint64_t v = __ballot(valid);
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
#pragma unroll
    for (int b = 0; b < kBits; ++b) {
        const uint32_t bit = (d >> b) & 1u;
        const uint64_t bm = __ballot(bit);
        const uint32_t s = 0u - bit;   // all ones where this lane's bit is set
        // keep the lanes whose bit equals ours: bm where set, ~bm where clear
        lo &= ~((uint32_t)bm ^ s);
        hi &= ~((uint32_t)(bm >> 32) ^ s);
    }
    return ((uint64_t)hi << 32) | lo;
}

template <int kBits, int kItems, typename KeyT>
__global__ __launch_bounds__(kBlock) void k_radix_hist(const KeyT* __restrict__ keys, PairCount cnt, int shift,
                                                       uint32_t* __restrict__ hist, int nblocks)
{
    constexpr int R = 1 << kBits;
    constexpr int kTile = kBlock * kItems;
    const uint64_t count = cnt.get();
    if ((uint64_t)blockIdx.x * kTile >= count) {
        // a workgroup past the keys (the grid is sized for the capacity)
        if (threadIdx.x < R) hist[(size_t)threadIdx.x * nblocks + blockIdx.x] = 0;
        return;
    }
    // 16 copies of the counts (per wave and lane % 4): a skewed digit, such as
    // the exponent byte of the depth keys, then meets at most 16 lanes of an
    // instruction on one counter
    __shared__ uint32_t h[16][R];
    for (int k = threadIdx.x; k < 16 * R; k += kBlock) (&h[0][0])[k] = 0;
    __syncthreads();
    const int copy = (threadIdx.x >> 6) * 4 + (threadIdx.x & 3);
    const uint64_t base = (uint64_t)blockIdx.x * kTile;
    // all loads first (one memory round trip), then the counts
    uint32_t k[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const uint64_t idx = base + (uint64_t)r * kBlock + threadIdx.x;
        k[r] = idx < count ? (uint32_t)keys[idx] : 0u;
    }
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
        const uint64_t idx = base + (uint64_t)r * kBlock + threadIdx.x;
        if (idx < count) atomicAdd(&h[copy][(k[r] >> shift) & (R - 1)], 1u);
    }
    __syncthreads();
    const int d = threadIdx.x;
    if (d < R) {
        uint32_t c = 0;
#pragma unroll
        for (int w = 0; w < 16; ++w) c += h[w][d];
        hist[(size_t)d * nblocks + blockIdx.x] = c;
    }
}

// One workgroup per digit: exclusive scan of that digit's counts over workgroups.
__global__ __launch_bounds__(kBlock) void k_radix_scan(uint32_t* __restrict__ hist, int nblocks,
                                                       uint32_t* __restrict__ digit_tot)
{
    __shared__ uint32_t lds4[4];
    uint32_t* row = hist + (size_t)blockIdx.x * nblocks;
    const int per = (nblocks + kBlock - 1) / kBlock;
    const int start = threadIdx.x * per;
    const int end = min(start + per, nblocks);
    uint32_t sum = 0;
    for (int k = start; k < end; ++k) sum += row[k];
    uint32_t total;
    uint32_t run = block_excl_scan(sum, lds4, &total);
    for (int k = start; k < end; ++k) {
        const uint32_t v = row[k];
        row[k] = run;
        run += v;
    }
    if (threadIdx.x == 0) digit_tot[blockIdx.x] = total;
}

template <int kBits, int kItems, typename KeyT, typename KeyOutT>
__global__ __launch_bounds__(kBlock) void k_radix_scatter(const KeyT* __restrict__ keys_in,
                                                          const uint32_t* __restrict__ vals_in, PairCount cnt,
                                                          int shift, const uint32_t* __restrict__ hist, int nblocks,
                                                          const uint32_t* __restrict__ digit_tot,
                                                          KeyOutT* __restrict__ keys_out,
                                                          uint32_t* __restrict__ vals_out,
                                                          const gs_splat* __restrict__ rect_src,
                                                          uint2* __restrict__ rect_out)
{
    constexpr int R = 1 << kBits;
    constexpr int kTile = kBlock * kItems;
    constexpr int kSlice = kTile / (kBlock / kWave);   // keys per wave
    __shared__ uint32_t wcnt[4][R];      // per-wave digit counts, then per-wave exclusive offsets
    __shared__ uint32_t gbase[R];        // global position of this workgroup's first key of each digit
    __shared__ uint32_t lstart[R];       // start of each digit in the workgroup's reordered keys
    __shared__ KeyT skey[kTile];
    __shared__ uint32_t sval[kTile];
    __shared__ uint32_t lds4[4];
    const uint64_t count = cnt.get();
    if ((uint64_t)blockIdx.x * kTile >= count) return;   // past the keys: nothing to move
    const int t = threadIdx.x, wave = t >> 6, lane = __lane_id();
    const uint32_t dt = t < R ? digit_tot[t] : 0u;
    const uint32_t dbase = block_excl_scan(dt, lds4, nullptr);
    if (t < R) {
        gbase[t] = dbase + hist[(size_t)t * nblocks + blockIdx.x];
        for (int w = 0; w < 4; ++w) wcnt[w][t] = 0;
    }
    __syncthreads();
    // rank within the wave's slice, in key order
    const uint64_t base = (uint64_t)blockIdx.x * kTile;
    const uint64_t wbase = base + (uint64_t)wave * kSlice;
    uint32_t key[kItems], val[kItems], rank[kItems];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const uint64_t idx = wbase + (uint64_t)i * kWave + lane;
        const bool valid = idx < count;
        key[i] = valid ? (uint32_t)keys_in[idx] : 0u;
        val[i] = valid ? (vals_in ? vals_in[idx] : (uint32_t)idx) : 0u;
    }
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const uint64_t idx = wbase + (uint64_t)i * kWave + lane;
        const bool valid = idx < count;
        const uint32_t d = (key[i] >> shift) & (R - 1);
        const uint64_t peers = match_digit<kBits>(d, valid);
        const uint32_t r = (uint32_t)__popcll(peers & lanemask_lt());
        const uint32_t pre = valid ? wcnt[wave][d] : 0u;
        rank[i] = pre + r;
        if (valid && r == 0) wcnt[wave][d] = pre + (uint32_t)__popcll(peers);
        // the next round reads counts this round's leaders wrote
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    uint32_t tot = 0;
    if (t < R) {
        for (int w = 0; w < 4; ++w) {
            const uint32_t c = wcnt[w][t];
            wcnt[w][t] = tot;
            tot += c;
        }
    }
    const uint32_t ls = block_excl_scan(t < R ? tot : 0u, lds4, nullptr);
    if (t < R) lstart[t] = ls;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
        const uint64_t idx = wbase + (uint64_t)i * kWave + lane;
        if (idx < count) {
            const uint32_t d = (key[i] >> shift) & (R - 1);
            const uint32_t lp = lstart[d] + wcnt[wave][d] + rank[i];
            skey[lp] = (KeyT)key[i];
            sval[lp] = val[i];
        }
    }
    __syncthreads();
    const uint32_t nvalid = (uint32_t)min((uint64_t)kTile, count - base);
    for (uint32_t j = t; j < nvalid; j += kBlock) {
        const uint32_t k = skey[j];
        const uint32_t d = (k >> shift) & (R - 1);
        const uint32_t pos = gbase[d] + (j - lstart[d]);
        const uint32_t v = sval[j];
        if (keys_out) keys_out[pos] = (KeyOutT)k;
        vals_out[pos] = v;
        if (rect_out) {
            // tile rectangle of Gaussian v in sorted order; culled Gaussians
            // (key ~0, no splat record) get an empty one
            uint2 r = make_uint2(0u, 0u);
            if (sizeof(KeyT) == 4 && k != 0xFFFFFFFFu) r = *reinterpret_cast<const uint2*>(reinterpret_cast<const uint32_t*>(rect_src + v) + kSplatRectWord);
            rect_out[pos] = r;
        }
    }
}

// One stable LSD pass over `bits` bits at `shift`; vals_in == nullptr means
// value = position, keys_out == nullptr drops the keys. The grids are sized
// for cnt.host keys (the capacity in device mode).
template <int kBits, int kItems, typename KeyT, typename KeyOutT>
void radix_pass_t(const KeyT* keys_in, const uint32_t* vals_in, PairCount cnt, int shift, KeyOutT* keys_out,
                  uint32_t* vals_out, uint32_t* hist, uint32_t* digit_tot, hipStream_t s,
                  const gs_splat* rect_src = nullptr, uint2* rect_out = nullptr)
{
    const int nblocks = (int)std::max<int64_t>(div_up((int64_t)cnt.host, (int64_t)kBlock * kItems), 1);
    hipLaunchKernelGGL((k_radix_hist<kBits, kItems, KeyT>), dim3(nblocks), dim3(kBlock), 0, s, keys_in, cnt, shift,
                       hist, nblocks);
    hipLaunchKernelGGL(k_radix_scan, dim3(1 << kBits), dim3(kBlock), 0, s, hist, nblocks, digit_tot);
    hipLaunchKernelGGL((k_radix_scatter<kBits, kItems, KeyT, KeyOutT>), dim3(nblocks), dim3(kBlock), 0, s, keys_in,
                       vals_in, cnt, shift,
                       hist, nblocks, digit_tot, keys_out, vals_out, rect_src, rect_out);
}

// A tile-sort pass over `bits` (1..8) bits, chosen at run time.
template <typename KeyT, typename KeyOutT>
hipError_t radix_pass(const KeyT* keys_in, const uint32_t* vals_in, PairCount cnt, int shift, int bits,
                      KeyOutT* keys_out, uint32_t* vals_out, uint32_t* hist, uint32_t* digit_tot, hipStream_t s)
{
    switch (bits) {
#define GS_PASS(b)                                                                                                   \
    case b:                                                                                                          \
        radix_pass_t<b, kPairItems>(keys_in, vals_in, cnt, shift, keys_out, vals_out, hist, digit_tot, s);        \
        break;
        GS_PASS(1) GS_PASS(2) GS_PASS(3) GS_PASS(4) GS_PASS(5) GS_PASS(6) GS_PASS(7) GS_PASS(8)
#undef GS_PASS
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---- pair offsets in depth order and pair emission ---------------------------

// Pairs emitted by each chunk of kDupChunk depth-ordered Gaussians.
__device__ __forceinline__ uint32_t rect_area(uint2 r)
{
    return ((r.y & 0xFFFFu) - (r.x & 0xFFFFu)) * ((r.y >> 16) - (r.x >> 16));
}

__global__ __launch_bounds__(kBlock) void k_pair_partial(const uint2* __restrict__ sorted_rect, int64_t n,
                                                         uint32_t* __restrict__ part)
{
    __shared__ uint32_t lds4[4];
    uint32_t sum = 0;
    for (int k = 0; k < kDupItems; ++k) {
        const int64_t i = (int64_t)blockIdx.x * kDupChunk + (int64_t)k * kBlock + threadIdx.x;
        if (i < n) sum += rect_area(sorted_rect[i]);
    }
    uint32_t total;
    block_excl_scan(sum, lds4, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

// Exclusive scan of the per-chunk totals (one workgroup).
__global__ __launch_bounds__(kBlock) void k_scan_partials(uint32_t* __restrict__ part, int count)
{
    __shared__ uint32_t lds4[4];
    const int per = (count + kBlock - 1) / kBlock;
    const int start = threadIdx.x * per, end = min(start + per, count);
    uint32_t sum = 0;
    for (int k = start; k < end; ++k) sum += part[k];
    uint32_t run = block_excl_scan(sum, lds4, nullptr);
    for (int k = start; k < end; ++k) {
        const uint32_t v = part[k];
        part[k] = run;
        run += v;
    }
}

// Inclusive maximum scan over the wave's lanes (DPP row shifts, then the row
// broadcasts); lanes without a source keep their value.
__device__ __forceinline__ int wave_max_scan(int v)
{
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x111, 0xF, 0xF, false));   // row_shr:1
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x112, 0xF, 0xF, false));   // row_shr:2
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x114, 0xF, 0xF, false));   // row_shr:4
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x118, 0xF, 0xF, false));   // row_shr:8
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x142, 0xA, 0xF, false));   // row_bcast:15
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x143, 0xC, 0xF, false));   // row_bcast:31
    return v;
}

__device__ __forceinline__ void wave_lds_fence()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Emits the (tile, Gaussian) pairs of a chunk of depth-ordered Gaussians, each
// Gaussian's tiles in row-major order of its rectangle. The chunk's offsets
// and rectangles are staged in LDS. Each wave then emits a contiguous quarter
// of the chunk's pairs, kDupWin consecutive pairs per round in groups of 64
// (consecutive lanes write consecutive addresses): the lanes mark in LDS where
// the Gaussians of the next kDupWin - 1 slots start inside the round's window
// (after its first pair, which belongs to the round's first Gaussian), and an
// inclusive maximum scan over the window gives each pair its Gaussian. Depth
// order puts every culled Gaussian (no tiles) after the visible ones, so starts
// inside a window are distinct.
constexpr int kDupGroups = 8;                   // 64-pair groups per round
constexpr int kDupWin = kWave * kDupGroups;     // pairs per round

template <typename KeyT>
__global__ __launch_bounds__(kBlock) void k_duplicate(const uint32_t* __restrict__ order,
                                                      const uint2* __restrict__ sorted_rect, int64_t n,
                                                      const uint32_t* __restrict__ part, int tiles_x,
                                                      PairCount pairs, KeyT* __restrict__ keys,
                                                      uint32_t* __restrict__ vals)
{
    // a device count beyond the capacity: no pair is emitted
    if (pairs.overflow()) return;
    const uint32_t capacity = (uint32_t)pairs.cap;
    __shared__ uint32_t soff[kDupChunk + 1];
    __shared__ uint32_t sgid[kDupChunk];
    __shared__ uint32_t sorg[kDupChunk];   // rectangle origin x0 | y0 << 16
    __shared__ uint32_t swid[kDupChunk];   // rectangle width in tiles
    __shared__ int smark[kBlock / kWave][kDupWin];
    __shared__ uint32_t lds4[4];
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kDupChunk;
    uint32_t cnt[kDupItems];
    uint32_t sum = 0;
    for (int k = 0; k < kDupItems; ++k) {
        const int slot = t * kDupItems + k;
        const int64_t i = base + slot;
        uint32_t c = 0, g = 0, org = 0, w = 1;
        if (i < n) {
            g = order[i];
            const uint2 r = sorted_rect[i];
            c = rect_area(r);
            if (c != 0) {
                org = r.x;
                w = (r.y & 0xFFFFu) - (r.x & 0xFFFFu);
            }
        }
        cnt[k] = c;
        sum += c;
        sgid[slot] = g;
        sorg[slot] = org;
        swid[slot] = w;
    }
    uint32_t total;
    uint32_t off = block_excl_scan(sum, lds4, &total);
    for (int k = 0; k < kDupItems; ++k) {
        soff[t * kDupItems + k] = off;
        off += cnt[k];
    }
    if (t == 0) soff[kDupChunk] = total;
    __syncthreads();
    const uint32_t gbase = part[blockIdx.x];
    const int wave = t >> 6, lane = __lane_id();
    const uint32_t q0 = (uint32_t)(((uint64_t)total * wave) / (kBlock / kWave));
    const uint32_t q1 = (uint32_t)(((uint64_t)total * (wave + 1)) / (kBlock / kWave));
    if (q0 >= q1) return;
    // last slot whose offset is <= q0 (the same address in every lane)
    int lo = 0, hi = kDupChunk;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (soff[mid] <= q0) lo = mid;
        else hi = mid;
    }
    int first = lo;
    int* mark = smark[wave];
    for (uint32_t p0 = q0; p0 < q1; p0 += kDupWin) {
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) mark[kWave * k + lane] = (k == 0 && lane == 0) ? 0 : -1;
        wave_lds_fence();
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            const int d = kWave * k + lane;   // slot offset from the round's first Gaussian
            const int sl = first + d;
            if (d > 0 && sl < kDupChunk) {
                const uint32_t o = soff[sl];
                if (o > p0 && o < p0 + kDupWin && soff[sl + 1] > o) mark[o - p0] = d;
            }
        }
        wave_lds_fence();
        // in stages, so each stage's LDS latency is paid once per round
        int m[kDupGroups];
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) m[k] = mark[kWave * k + lane];
        int run = 0;   // owner of the window's positions so far (mark[0] = 0)
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            m[k] = max(wave_max_scan(m[k]), run);
            run = __builtin_amdgcn_readlane(m[k], kWave - 1);
        }
        uint32_t o[kDupGroups], w[kDupGroups], org[kDupGroups], gid[kDupGroups];
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            const int slot = first + m[k];
            o[k] = soff[slot];
            w[k] = swid[slot];
            org[k] = sorg[slot];
            gid[k] = sgid[slot];
        }
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            const uint32_t p = p0 + kWave * k + lane;
            const uint32_t i = p - o[k];
            const uint32_t q = i / w[k];
            const uint32_t tx = (org[k] & 0xFFFFu) + (i - q * w[k]);
            const uint32_t ty = (org[k] >> 16) + q;
            const uint32_t out = gbase + p;
            // only a num_pairs that disagrees with the preprocess gets past the capacity
            if (p < q1 && out < capacity) {
                keys[out] = (KeyT)(ty * (uint32_t)tiles_x + tx);
                vals[out] = gid[k];
            }
        }
        // the next round starts with the Gaussian holding pair p0 + kDupWin: the
        // window's last owner, or the one after it if that ends exactly there
        const int last = first + run;
        first = last + (soff[last + 1] == p0 + kDupWin ? 1 : 0);
        wave_lds_fence();   // this round's mark reads before the next round's clear
    }
}

// One wave per tile boundary v = 0..n_tiles: the first position whose tile id
// is >= v, by a 64-way search. Each round the lanes probe 64 evenly spaced
// positions of [lo, hi); the probes below v form a prefix (the keys are
// sorted), so their count c narrows the answer to (probe c-1, probe c]. About
// log64(P) dependent loads instead of log2(P). Boundary v ends tile v - 1 and
// starts tile v.
template <typename KeyT>
__global__ __launch_bounds__(kBlock) void k_ranges(const KeyT* __restrict__ sorted_tiles, PairCount pairs,
                                                   int n_tiles, uint32_t* __restrict__ ranges)
{
    const uint32_t count = (uint32_t)pairs.get();
    const int v = (int)blockIdx.x * (kBlock / kWave) + (int)(threadIdx.x >> 6);
    if (v > n_tiles) return;
    const uint32_t lane = __lane_id();
    uint32_t lo = 0, hi = count;   // the answer lies in [lo, hi]
    while (hi > lo) {
        const uint32_t step = (hi - lo + kWave - 1) / kWave;
        const uint32_t p = lo + lane * step;
        const bool below = p < hi && (uint32_t)sorted_tiles[p] < (uint32_t)v;
        const uint32_t c = (uint32_t)__popcll(__ballot(below));
        const uint32_t nlo = c ? lo + (c - 1) * step + 1 : lo;
        hi = min(hi, lo + c * step);
        lo = nlo;
    }
    if (lane == 0) {
        if (v < n_tiles) ranges[2 * v] = lo;
        if (v > 0) ranges[2 * v - 1] = lo;
    }
}

}  // namespace

hipError_t launch_depth_sort(int64_t n, const uint32_t* depth_key, const gs_splat* splats, const Workspace& ws,
                             const uint32_t** order_out, hipStream_t s)
{
    const uint32_t* kin = depth_key;
    const uint32_t* vin = nullptr;
    uint32_t* kbuf[2] = {ws.keys_a, ws.keys_b};
    uint32_t* vbuf[2] = {ws.vals_a, ws.vals_b};
    const PairCount keys_n{nullptr, (uint64_t)n, (uint64_t)n};
    for (int p = 0; p < 4; ++p) {
        const bool last = p == 3;
        uint32_t* kout = last ? nullptr : kbuf[p & 1];
        if (last)
            radix_pass_t<8, kSortItems>(kin, vin, keys_n, 8 * p, (uint32_t*)nullptr, vbuf[p & 1], ws.hist,
                                        ws.digit_tot + kRadix * p, s, splats, ws.sorted_rect);
        else
            radix_pass_t<8, kSortItems>(kin, vin, keys_n, 8 * p, kout, vbuf[p & 1], ws.hist,
                                        ws.digit_tot + kRadix * p, s);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        kin = kbuf[p & 1];
        vin = vbuf[p & 1];
    }
    *order_out = vin;
    return hipSuccess;
}

hipError_t launch_pair_offsets(int64_t n, const Workspace& ws, hipStream_t s)
{
    const int nb = (int)div_up(n, kDupChunk);
    hipLaunchKernelGGL(k_pair_partial, dim3(nb), dim3(kBlock), 0, s, ws.sorted_rect, n, ws.scan_part);
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kBlock), 0, s, ws.scan_part, nb);
    return hipGetLastError();
}

hipError_t launch_duplicate(const Cam& cam, int64_t n, const uint32_t* order, const Workspace& ws,
                            PairCount pairs, TileKeys keys_out, uint32_t* vals_out, hipStream_t s)
{
    const int nb = (int)div_up(n, kDupChunk);
    if (keys_out.narrow)
        hipLaunchKernelGGL(k_duplicate<uint16_t>, dim3(nb), dim3(kBlock), 0, s, order, ws.sorted_rect, n, ws.scan_part,
                           cam.tiles_x, pairs, static_cast<uint16_t*>(keys_out.p), vals_out);
    else
        hipLaunchKernelGGL(k_duplicate<uint32_t>, dim3(nb), dim3(kBlock), 0, s, order, ws.sorted_rect, n, ws.scan_part,
                           cam.tiles_x, pairs, static_cast<uint32_t*>(keys_out.p), vals_out);
    return hipGetLastError();
}

// Bits of the tile id, and how they are split over passes of at most 8 bits.
static int tile_bits(const Cam& cam)
{
    const uint32_t n_tiles = (uint32_t)cam.tiles_x * (uint32_t)cam.tiles_y;
    int bits = 0;
    while (bits < 32 && ((n_tiles - 1) >> bits) != 0) ++bits;
    return bits;
}

int tile_sort_passes(const Cam& cam) { return (tile_bits(cam) + 7) / 8; }

bool tile_keys_narrow(const Cam& cam) { return (int64_t)cam.tiles_x * cam.tiles_y <= 65536; }

template <typename KeyT>
static hipError_t tile_sort_t(const Cam& cam, PairCount num_pairs, const Workspace& ws, uint32_t* values,
                              uint32_t* tile_ids_out, TileKeys* sorted_tiles, hipStream_t s)
{
    const int bits = tile_bits(cam);
    const int passes = (bits + 7) / 8;
    KeyT* kbuf[2] = {reinterpret_cast<KeyT*>(ws.pair_keys_a), reinterpret_cast<KeyT*>(ws.pair_keys_b)};
    uint32_t* vbuf[2] = {ws.pair_vals_a, ws.pair_vals_b};
    int src = 0, shift = 0;
    for (int p = 0; p < passes; ++p) {
        const bool last = p == passes - 1;
        const int pb = (bits - shift + (passes - p) - 1) / (passes - p);   // remaining bits spread evenly
        uint32_t* vout = last ? values : vbuf[src ^ 1];
        hipError_t e;
        if (last && tile_ids_out) {
            // the caller's 32-bit tile ids double as the sorted keys for the ranges
            e = radix_pass(kbuf[src], vbuf[src], num_pairs, shift, pb, tile_ids_out, vout, ws.hist, ws.digit_tot, s);
            *sorted_tiles = TileKeys{tile_ids_out, false};
        }
        else {
            e = radix_pass(kbuf[src], vbuf[src], num_pairs, shift, pb, kbuf[src ^ 1], vout, ws.hist, ws.digit_tot, s);
            if (last) *sorted_tiles = TileKeys{kbuf[src ^ 1], sizeof(KeyT) == 2};
        }
        if (e != hipSuccess) return e;
        shift += pb;
        src ^= 1;
    }
    return hipSuccess;
}

hipError_t launch_tile_sort(const Cam& cam, PairCount num_pairs, const Workspace& ws, uint32_t* values,
                            uint32_t* tile_ids_out, TileKeys* sorted_tiles, hipStream_t s)
{
    return tile_keys_narrow(cam) ? tile_sort_t<uint16_t>(cam, num_pairs, ws, values, tile_ids_out, sorted_tiles, s)
                                 : tile_sort_t<uint32_t>(cam, num_pairs, ws, values, tile_ids_out, sorted_tiles, s);
}

hipError_t launch_ranges(const Cam& cam, PairCount num_pairs, TileKeys sorted_tiles, uint32_t* tile_ranges,
                         hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const dim3 grid((unsigned)div_up(n_tiles + 1, kBlock / kWave));
    if (sorted_tiles.narrow)
        hipLaunchKernelGGL(k_ranges<uint16_t>, grid, dim3(kBlock), 0, s, static_cast<const uint16_t*>(sorted_tiles.p),
                           num_pairs, n_tiles, tile_ranges);
    else
        hipLaunchKernelGGL(k_ranges<uint32_t>, grid, dim3(kBlock), 0, s, static_cast<const uint32_t*>(sorted_tiles.p),
                           num_pairs, n_tiles, tile_ranges);
    return hipGetLastError();
}

}  // namespace gsr
