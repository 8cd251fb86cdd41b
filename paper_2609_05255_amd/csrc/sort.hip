// Depth-sorted per-tile lists (Sec. 3.1 "depth-sorted order"): the pairs must
// come out ordered by (tile, depth key, Gaussian index).
//
// Instead of radix-sorting P 45-bit (tile, depth) keys, the Gaussians are
// sorted once by depth (4 stable 8-bit LSD passes over n 32-bit keys with the
// index as value, so equal depths stay in index order). Then, in that order,
// each Gaussian gets one entry per 4x4-tile block its rectangle meets (about a
// quarter as many entries as pairs), a stable LSD sort on the block id groups
// the entries by block with depth order kept inside each block, and every
// block's 16 tile lists are cut out of its entries by ordered (ballot)
// compaction, each list written once, at its final place.
//
// One radix pass = k_radix_hist (per-workgroup digit counts) + k_radix_scan
// (exclusive offsets per digit over workgroups) + k_radix_scatter: each wave
// ranks a contiguous slice of the workgroup's keys with ballot-matched digits
// (no workgroup barrier per round), the workgroup reorders its 4096 keys by
// digit in LDS, and writes each digit's run to consecutive global addresses.
// The grids are sized for the most keys a call can meet (the capacity, for
// the block entries); workgroups past the device-side count do nothing, and
// the scan reads only the workgroups below it. A single-pass block sort's
// scatter has one workgroup more, which writes the tile lists' segment table
// from that pass's digit totals (the blocks' entry counts).
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
    if ((uint64_t)blockIdx.x * kTile >= count) return;   // past the keys: the scan does not read it
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
    for (int d = threadIdx.x; d < R; d += kBlock) {
        uint32_t c = 0;
#pragma unroll
        for (int w = 0; w < 16; ++w) c += h[w][d];
        hist[(size_t)d * nblocks + blockIdx.x] = c;
    }
}

// One workgroup per digit: exclusive scan of that digit's counts over the
// workgroups that hold keys (the first ceil(count / tile) of the nblocks).
__global__ __launch_bounds__(kBlock) void k_radix_scan(uint32_t* __restrict__ hist, int nblocks, PairCount cnt,
                                                       int tile, uint32_t* __restrict__ digit_tot)
{
    __shared__ uint32_t lds4[4];
    uint32_t* row = hist + (size_t)blockIdx.x * nblocks;
    const int active = (int)min((uint64_t)nblocks, (cnt.get() + (uint64_t)tile - 1) / (uint64_t)tile);
    const int per = (active + kBlock - 1) / kBlock;
    const int start = threadIdx.x * per;
    const int end = min(start + per, active);
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

// The block entries' segment table (see k_segments), written by one extra
// workgroup of the block sort's scatter from that pass's digit totals.
struct SegTable {
    uint32_t* block_ranges;   // nullptr: no table
    uint32_t* seg_base;
    uint32_t* seg_block;
    uint32_t* counters;
    int n_blocks;
};

__device__ void segment_table_256(const uint32_t* __restrict__ block_count, const SegTable& t);

template <int kBits, int kItems, typename KeyT, typename KeyOutT>
__global__ __launch_bounds__(kBlock) void k_radix_scatter(const KeyT* __restrict__ keys_in,
                                                          const uint32_t* __restrict__ vals_in, PairCount cnt,
                                                          int shift, const uint32_t* __restrict__ hist, int nblocks,
                                                          const uint32_t* __restrict__ digit_tot,
                                                          KeyOutT* __restrict__ keys_out,
                                                          uint32_t* __restrict__ vals_out,
                                                          const gs_splat* __restrict__ rect_src,
                                                          uint2* __restrict__ rect_out, SegTable seg)
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
    if (seg.block_ranges && blockIdx.x == gridDim.x - 1) {   // the extra workgroup
        segment_table_256(digit_tot, seg);
        return;
    }
    const uint64_t count = cnt.get();
    if ((uint64_t)blockIdx.x * kTile >= count) return;   // past the keys: nothing to move
    const int t = threadIdx.x, wave = t >> 6, lane = __lane_id();
    // digits t * kDPT + j (consecutive per thread)
    constexpr int kDPT = R > kBlock ? R / kBlock : 1;
    uint32_t dtv[kDPT], dsum = 0;
#pragma unroll
    for (int j = 0; j < kDPT; ++j) {
        const int d = t * kDPT + j;
        dtv[j] = d < R ? digit_tot[d] : 0u;
        dsum += dtv[j];
    }
    uint32_t dbase = block_excl_scan(dsum, lds4, nullptr);
#pragma unroll
    for (int j = 0; j < kDPT; ++j) {
        const int d = t * kDPT + j;
        if (d < R) {
            gbase[d] = dbase + hist[(size_t)d * nblocks + blockIdx.x];
            for (int w = 0; w < 4; ++w) wcnt[w][d] = 0;
        }
        dbase += dtv[j];
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
    uint32_t tots[kDPT], tsum = 0;
#pragma unroll
    for (int j = 0; j < kDPT; ++j) {
        const int d = t * kDPT + j;
        uint32_t tot = 0;
        if (d < R) {
            for (int w = 0; w < 4; ++w) {
                const uint32_t c = wcnt[w][d];
                wcnt[w][d] = tot;
                tot += c;
            }
        }
        tots[j] = tot;
        tsum += tot;
    }
    uint32_t ls = block_excl_scan(tsum, lds4, nullptr);
#pragma unroll
    for (int j = 0; j < kDPT; ++j) {
        const int d = t * kDPT + j;
        if (d < R) lstart[d] = ls;
        ls += tots[j];
    }
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
                  const gs_splat* rect_src = nullptr, uint2* rect_out = nullptr,
                  SegTable seg = SegTable{nullptr, nullptr, nullptr, nullptr, 0})
{
    const int nblocks = (int)std::max<int64_t>(div_up((int64_t)cnt.host, (int64_t)kBlock * kItems), 1);
    hipLaunchKernelGGL((k_radix_hist<kBits, kItems, KeyT>), dim3(nblocks), dim3(kBlock), 0, s, keys_in, cnt, shift,
                       hist, nblocks);
    hipLaunchKernelGGL(k_radix_scan, dim3(1 << kBits), dim3(kBlock), 0, s, hist, nblocks, cnt, kBlock * kItems,
                       digit_tot);
    hipLaunchKernelGGL((k_radix_scatter<kBits, kItems, KeyT, KeyOutT>), dim3(nblocks + (seg.block_ranges ? 1 : 0)),
                       dim3(kBlock), 0, s, keys_in, vals_in, cnt, shift, hist, nblocks, digit_tot, keys_out, vals_out,
                       rect_src, rect_out, seg);
}

// A block-sort pass over `bits` (1..9) bits, 8192 keys per workgroup: twice
// the depth sort's, for longer runs per digit among the 9-bit digits.
constexpr int kBlockSortBits = 9;
hipError_t block_radix_pass(const uint32_t* keys_in, const uint32_t* vals_in, PairCount cnt, int shift, int bits,
                            uint32_t* keys_out, uint32_t* vals_out, uint32_t* hist, uint32_t* digit_tot, hipStream_t s,
                            SegTable seg)
{
    switch (bits) {
#define GS_PASS(b)                                                                                                   \
    case b:                                                                                                          \
        radix_pass_t<b, kBlockSortItems>(keys_in, vals_in, cnt, shift, keys_out, vals_out, hist, digit_tot, s,     \
                                         nullptr, nullptr, seg);                                                     \
        break;
        GS_PASS(1) GS_PASS(2) GS_PASS(3) GS_PASS(4) GS_PASS(5) GS_PASS(6) GS_PASS(7) GS_PASS(8) GS_PASS(9)
#undef GS_PASS
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---- block entries in depth order -------------------------------------------
//
// A block is kBlockDim x kBlockDim tiles. Each visible Gaussian gets one entry
// per block its tile rectangle meets, in depth order; the entries are then
// sorted by block id (stable, so depth order holds inside a block), and each
// block's tile lists are cut out of its entries by ordered compaction.

// Area of a packed rectangle (x0 | y0 << 16, x1 | y1 << 16, half-open).
__device__ __forceinline__ uint32_t rect_area(uint2 r)
{
    return ((r.y & 0xFFFFu) - (r.x & 0xFFFFu)) * ((r.y >> 16) - (r.x >> 16));
}

// Block rectangle (half-open, block units, packed like a tile rectangle) of a
// tile rectangle; an empty rectangle stays empty.
__device__ __forceinline__ uint2 block_rect(uint2 r)
{
    if (rect_area(r) == 0) return make_uint2(0u, 0u);
    const uint32_t x0 = r.x & 0xFFFFu, y0 = r.x >> 16, x1 = r.y & 0xFFFFu, y1 = r.y >> 16;
    constexpr uint32_t kS = 2, kR = kBlockDim - 1;   // log2 and mask of the block size
    static_assert(kBlockDim == 1 << kS, "block size");
    return make_uint2((x0 >> kS) | ((y0 >> kS) << 16), ((x1 + kR) >> kS) | (((y1 + kR) >> kS) << 16));
}

// Entries of each chunk of kDupChunk depth-ordered Gaussians.
__global__ __launch_bounds__(kBlock) void k_entry_partial(const uint2* __restrict__ sorted_rect, int64_t n,
                                                          uint32_t* __restrict__ part)
{
    __shared__ uint32_t lds4[4];
    uint32_t sum = 0;
    for (int k = 0; k < kDupItems; ++k) {
        const int64_t i = (int64_t)blockIdx.x * kDupChunk + (int64_t)k * kBlock + threadIdx.x;
        if (i < n) sum += rect_area(block_rect(sorted_rect[i]));
    }
    uint32_t total;
    block_excl_scan(sum, lds4, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

// Exclusive scan of the per-chunk totals (one workgroup); the grand total, the
// number of entries, goes to *entries (0 when the pair count is over capacity:
// nothing downstream then reads an entry).
__global__ __launch_bounds__(kBlock) void k_scan_partials(uint32_t* __restrict__ part, int count, PairCount pairs,
                                                          uint64_t* __restrict__ entries)
{
    __shared__ uint32_t lds4[4];
    const int per = (count + kBlock - 1) / kBlock;
    const int start = threadIdx.x * per, end = min(start + per, count);
    uint32_t sum = 0;
    for (int k = start; k < end; ++k) sum += part[k];
    uint32_t total;
    uint32_t run = block_excl_scan(sum, lds4, &total);
    for (int k = start; k < end; ++k) {
        const uint32_t v = part[k];
        part[k] = run;
        run += v;
    }
    if (threadIdx.x == 0) *entries = pairs.overflow() ? 0ull : (uint64_t)total;
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

// Bit 4k + i set where the tile rectangle r meets tile (4 bx + i, 4 by + k).
__device__ __forceinline__ uint32_t tile_mask(uint2 r, int bx, int by)
{
    const int ox = kBlockDim * bx, oy = kBlockDim * by;
    const int cx0 = max((int)(r.x & 0xFFFFu) - ox, 0), cx1 = min((int)(r.y & 0xFFFFu) - ox, kBlockDim);
    const int cy0 = max((int)(r.x >> 16) - oy, 0), cy1 = min((int)(r.y >> 16) - oy, kBlockDim);
    if (cx1 <= cx0 || cy1 <= cy0) return 0u;
    const uint32_t cols = ((1u << cx1) - 1u) & ~((1u << cx0) - 1u);
    const uint32_t rows = ((1u << cy1) - 1u) & ~((1u << cy0) - 1u);
    // rows bit k -> bit 4k, then one copy of the column bits per row
    const uint32_t spread = (rows & 1u) | ((rows & 2u) << 3) | ((rows & 4u) << 6) | ((rows & 8u) << 9);
    return cols * spread;
}

// Emits the entries of a chunk of depth-ordered Gaussians, each Gaussian's
// blocks in row-major order of its block rectangle: key = block id << 16 |
// the mask of the block's tiles that the Gaussian's rectangle meets, value =
// the Gaussian's index. The chunk's offsets, rectangles and indices are staged
// in LDS. Each wave then emits a contiguous quarter of the chunk's entries,
// kDupWin consecutive entries per round in groups of 64 (consecutive lanes
// write consecutive addresses): the lanes mark in LDS where the Gaussians of
// the next kDupWin - 1 slots start inside the round's window (after its first
// entry, which belongs to the round's first Gaussian), and an inclusive
// maximum scan over the window gives each entry its Gaussian. Depth order puts
// every culled Gaussian (no tiles) after the visible ones, so starts inside a
// window are distinct.
constexpr int kDupGroups = 8;                   // 64-entry groups per round
constexpr int kDupWin = kWave * kDupGroups;     // entries per round
constexpr int kMaskBits = 16;                   // low key bits: the tile mask

__global__ __launch_bounds__(kBlock) void k_block_entries(const uint32_t* __restrict__ order,
                                                          const uint2* __restrict__ sorted_rect, int64_t n,
                                                          const uint32_t* __restrict__ part, int blocks_x,
                                                          PairCount entries, uint32_t* __restrict__ keys,
                                                          uint32_t* __restrict__ vals)
{
    const uint32_t count = (uint32_t)entries.get();   // 0 when the pairs are over capacity
    __shared__ uint32_t soff[kDupChunk + 1];
    __shared__ uint32_t sorg[kDupChunk];   // block rectangle origin x0 | y0 << 16
    __shared__ uint32_t swid[kDupChunk];   // block rectangle width
    __shared__ uint2 srect[kDupChunk];     // tile rectangle
    __shared__ uint32_t sgid[kDupChunk];   // Gaussian index
    __shared__ int smark[kBlock / kWave][kDupWin];
    __shared__ uint32_t lds4[4];
    const int t = threadIdx.x;
    const int64_t base = (int64_t)blockIdx.x * kDupChunk;
    uint32_t cnt[kDupItems];
    uint32_t sum = 0;
    for (int k = 0; k < kDupItems; ++k) {
        const int slot = t * kDupItems + k;
        const int64_t i = base + slot;
        uint32_t c = 0, org = 0, w = 1, g = 0;
        uint2 tr = make_uint2(0u, 0u);
        if (i < n) {
            tr = sorted_rect[i];
            g = order[i];
            const uint2 r = block_rect(tr);
            c = rect_area(r);
            if (c != 0) {
                org = r.x;
                w = (r.y & 0xFFFFu) - (r.x & 0xFFFFu);
            }
        }
        cnt[k] = c;
        sum += c;
        sorg[slot] = org;
        swid[slot] = w;
        srect[slot] = tr;
        sgid[slot] = g;
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
        uint2 tr[kDupGroups];
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            const int slot = first + m[k];
            o[k] = soff[slot];
            w[k] = swid[slot];
            org[k] = sorg[slot];
            tr[k] = srect[slot];
            gid[k] = sgid[slot];
        }
#pragma unroll
        for (int k = 0; k < kDupGroups; ++k) {
            const uint32_t p = p0 + kWave * k + lane;
            const uint32_t i = p - o[k];
            // i / w by a float reciprocal, corrected to the exact quotient (an
            // entry index and a block-rectangle width are both below 2^16, so
            // the estimate is off by at most one)
            uint32_t q = (uint32_t)((float)i * __builtin_amdgcn_rcpf((float)w[k]));
            q = q * w[k] > i ? q - 1u : q;
            q = (q + 1u) * w[k] <= i ? q + 1u : q;
            const uint32_t bx = (org[k] & 0xFFFFu) + (i - q * w[k]);
            const uint32_t by = (org[k] >> 16) + q;
            const uint32_t out = gbase + p;
            // a count of 0 (pairs over capacity) writes nothing
            if (p < q1 && out < count) {
                keys[out] = ((by * (uint32_t)blocks_x + bx) << kMaskBits) | tile_mask(tr[k], (int)bx, (int)by);
                vals[out] = gid[k];
            }
        }
        // the next round starts with the Gaussian holding entry p0 + kDupWin: the
        // window's last owner, or the one after it if that ends exactly there
        const int last = first + run;
        first = last + (soff[last + 1] == p0 + kDupWin ? 1 : 0);
        wave_lds_fence();   // this round's mark reads before the next round's clear
    }
}

// One wave per boundary v = 0..n_keys of sorted keys: the first position whose
// key >> shift is >= v, by a 64-way search. Each round the lanes probe 64 evenly spaced
// positions of [lo, hi); the probes below v form a prefix (the keys are
// sorted), so their count c narrows the answer to (probe c-1, probe c]. About
// log64(count) dependent loads instead of log2(count). Boundary v ends range
// v - 1 and starts range v.
__global__ __launch_bounds__(kBlock) void k_ranges(const uint32_t* __restrict__ sorted_keys, int shift,
                                                   PairCount cnt, int n_keys, uint32_t* __restrict__ ranges)
{
    const uint32_t count = (uint32_t)cnt.get();
    const int v = (int)blockIdx.x * (kBlock / kWave) + (int)(threadIdx.x >> 6);
    if (v > n_keys) return;
    const uint32_t lane = __lane_id();
    uint32_t lo = 0, hi = count;   // the answer lies in [lo, hi]
    while (hi > lo) {
        const uint32_t step = (hi - lo + kWave - 1) / kWave;
        const uint32_t p = lo + lane * step;
        const bool below = p < hi && (sorted_keys[p] >> shift) < (uint32_t)v;
        const uint32_t c = (uint32_t)__popcll(__ballot(below));
        const uint32_t nlo = c ? lo + (c - 1) * step + 1 : lo;
        hi = min(hi, lo + c * step);
        lo = nlo;
    }
    if (lane == 0) {
        if (v < n_keys) ranges[2 * v] = lo;
        if (v > 0) ranges[2 * v - 1] = lo;
    }
}

// ---- tile lists out of the block entries ------------------------------------
//
// Each block's entries are cut into segments of kSegEntries, one workgroup
// per segment and one sub-segment of 512 entries per wave. k_tile_count
// counts, per sub-segment, the entries that meet each of the block's 16 tiles;
// k_tile_scan turns the counts into each sub-segment's offset inside each
// tile's list and each tile's length; k_tile_starts places the lists in tile
// order (the ranges); k_tile_emit writes every tile's Gaussians, in entry
// order, by ballot compaction.

constexpr int kBlockTiles = kBlockDim * kBlockDim;             // 16
constexpr int kSegRounds = 8;                                  // 64-entry rounds per wave
constexpr int kSegEntries = kSegRounds * kBlock;               // 2048 entries per segment
constexpr int kSubSegs = kBlock / kWave;                       // one sub-segment per wave
constexpr int kListThreads = 1024;                             // single-workgroup scans
static_assert(kBlockTiles == 16, "tile masks are 16 bits");

// Exclusive scan of one value per thread over a 1024-thread workgroup.
template <typename T>
__device__ __forceinline__ T wg_excl_scan_1024(T v, T* lds16, T* total)
{
    const int lane = __lane_id(), wave = threadIdx.x >> 6;
    T x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const T y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) lds16[wave] = x;
    __syncthreads();
    T before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kListThreads / kWave; ++w) {
        const T s = lds16[w];
        if (w < wave) before += s;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return before + x - v;
}

// Segment table: one workgroup. seg_base[b] = first segment of block b (and
// seg_base[n_blocks] = their number), seg_block[s] = the block of segment s,
// counters[0] = the number of segments.
__global__ __launch_bounds__(kListThreads) void k_segments(const uint32_t* __restrict__ block_count,
                                                           uint32_t* __restrict__ block_ranges, int n_blocks,
                                                           uint32_t* __restrict__ seg_base,
                                                           uint32_t* __restrict__ seg_block,
                                                           uint32_t* __restrict__ counters)
{
    __shared__ uint32_t lds16[kListThreads / kWave];
    uint32_t carry = 0, ecarry = 0;
    for (int b0 = 0; b0 < n_blocks; b0 += kListThreads) {
        const int b = b0 + (int)threadIdx.x;
        uint32_t len = 0;
        if (block_count) {
            // the ranges follow from the counts (a single-pass block sort's digit totals)
            len = b < n_blocks ? block_count[b] : 0u;
            uint32_t etotal;
            const uint32_t start = ecarry + wg_excl_scan_1024(len, lds16, &etotal);
            if (b < n_blocks) {
                block_ranges[2 * b] = start;
                block_ranges[2 * b + 1] = start + len;
            }
            ecarry += etotal;
        } else if (b < n_blocks) {
            len = block_ranges[2 * b + 1] - block_ranges[2 * b];
        }
        const uint32_t ns = (len + kSegEntries - 1) / kSegEntries;
        uint32_t total;
        const uint32_t first = carry + wg_excl_scan_1024(ns, lds16, &total);
        if (b < n_blocks) {
            seg_base[b] = first;
            for (uint32_t k = 0; k < ns; ++k) seg_block[first + k] = (uint32_t)b;
        }
        carry += total;
    }
    if (threadIdx.x == 0) {
        seg_base[n_blocks] = carry;
        counters[0] = carry;
    }
}

// k_segments' table from the digit totals of a single-pass block sort, for
// one 256-thread workgroup (the block sort scatter's extra one).
__device__ void segment_table_256(const uint32_t* __restrict__ block_count, const SegTable& t)
{
    __shared__ uint32_t lds4s[4];
    uint32_t carry = 0, ecarry = 0;
    for (int b0 = 0; b0 < t.n_blocks; b0 += kBlock) {
        const int b = b0 + (int)threadIdx.x;
        const uint32_t len = b < t.n_blocks ? block_count[b] : 0u;
        uint32_t etotal, total;
        const uint32_t start = ecarry + block_excl_scan(len, lds4s, &etotal);
        const uint32_t ns = (len + kSegEntries - 1) / kSegEntries;
        const uint32_t first = carry + block_excl_scan(ns, lds4s, &total);
        if (b < t.n_blocks) {
            t.block_ranges[2 * b] = start;
            t.block_ranges[2 * b + 1] = start + len;
            t.seg_base[b] = first;
            for (uint32_t k = 0; k < ns; ++k) t.seg_block[first + k] = (uint32_t)b;
        }
        ecarry += etotal;
        carry += total;
    }
    if (threadIdx.x == 0) {
        t.seg_base[t.n_blocks] = carry;
        t.counters[0] = carry;
    }
}

// The entry range of segment s: block b, entries [e0, e1).
struct Segment {
    uint32_t b, e0, e1;
};

__device__ __forceinline__ Segment segment_of(uint32_t s, const uint32_t* __restrict__ seg_block,
                                              const uint32_t* __restrict__ seg_base,
                                              const uint32_t* __restrict__ block_ranges)
{
    Segment g;
    g.b = seg_block[s];
    const uint32_t j = s - seg_base[g.b];
    const uint32_t end = block_ranges[2 * g.b + 1];
    g.e0 = block_ranges[2 * g.b] + j * (uint32_t)kSegEntries;
    g.e1 = min(g.e0 + (uint32_t)kSegEntries, end);
    return g;
}

// The tile masks (and, for the emission, the Gaussian indices) of this wave's
// kSegRounds x 64 entries of the segment; lanes past the segment get mask 0.
// All loads are issued together, at indices clamped into the segment.
template <bool kIds>
__device__ __forceinline__ void load_segment(const Segment& g, const uint32_t* __restrict__ ent_key,
                                             const uint32_t* __restrict__ ent_gid, uint32_t mask[kSegRounds],
                                             uint32_t gid[kSegRounds])
{
    const uint32_t w0 = g.e0 + (threadIdx.x >> 6) * (kSegRounds * kWave) + __lane_id();
    const uint32_t last = g.e1 - 1u;   // segments are never empty
#pragma unroll
    for (int r = 0; r < kSegRounds; ++r) {
        const uint32_t e = min(w0 + r * kWave, last);
        mask[r] = ent_key[e];
        if (kIds) gid[r] = ent_gid[e];
    }
#pragma unroll
    for (int r = 0; r < kSegRounds; ++r)
        mask[r] = w0 + r * kWave <= last ? mask[r] & ((1u << kMaskBits) - 1u) : 0u;
}

// k_tile_count: per wave (a sub-segment of kSegRounds x 64 entries), the
// entries meeting each tile of the block; lane l (< 16) writes the count of
// tile l to wave_cnt[(4 s + wave) * 16 + l]. Tile-major, so that a single count
// is live at a time.
__global__ __launch_bounds__(kBlock) void k_tile_count(const uint32_t* __restrict__ ent_key,
                                                       const uint32_t* __restrict__ block_ranges,
                                                       const uint32_t* __restrict__ seg_base,
                                                       const uint32_t* __restrict__ seg_block,
                                                       const uint32_t* __restrict__ counters,
                                                       uint32_t* __restrict__ wave_cnt)
{
    const uint32_t s = blockIdx.x;
    if (s >= counters[0]) return;
    const Segment g = segment_of(s, seg_block, seg_base, block_ranges);
    uint32_t mask[kSegRounds], gid[kSegRounds];
    load_segment<false>(g, ent_key, nullptr, mask, gid);
    const int lane = __lane_id();
    uint32_t mine = 0;
#pragma unroll
    for (int l = 0; l < kBlockTiles; ++l) {
        uint32_t c = 0;
#pragma unroll
        for (int r = 0; r < kSegRounds; ++r) c += (uint32_t)__popcll(__ballot((mask[r] >> l) & 1u));
        // c is uniform: take it as such before the per-lane select
        mine = lane == l ? (uint32_t)__builtin_amdgcn_readfirstlane(c) : mine;
    }
    if (lane < kBlockTiles) wave_cnt[((size_t)s * kSubSegs + (threadIdx.x >> 6)) * kBlockTiles + lane] = mine;
}

// One wave per block: lane 16 q + l holds tile l of the q-th quarter of the
// block's sub-segments (4 per segment, in entry order): it sums its quarter's
// counts (loads issued together), the quarters are scanned across q, and a
// second sweep turns wave_cnt into each sub-segment's exclusive offset inside
// the tile's list. The tile's length goes to tile_ranges[2 t + 1].
__global__ __launch_bounds__(kWave) void k_tile_scan(const uint32_t* __restrict__ seg_base, int n_blocks,
                                                     int blocks_x, int tiles_x, int tiles_y,
                                                     uint32_t* __restrict__ wave_cnt, uint32_t* __restrict__ tile_ranges)
{
    const int b = blockIdx.x;
    if (b >= n_blocks) return;
    const int lane = __lane_id(), q = lane >> 4, l = lane & 15;
    const uint32_t s0 = seg_base[b] * kSubSegs, s1 = seg_base[b + 1] * kSubSegs;
    const uint32_t per = (s1 - s0 + 3) / 4;
    const uint32_t a0 = min(s0 + per * q, s1), a1 = min(a0 + per, s1);
    uint32_t sum = 0;
    for (uint32_t sb = a0; sb < a1; sb += 8) {
        uint32_t v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = sb + k < a1 ? wave_cnt[(size_t)(sb + k) * kBlockTiles + l] : 0u;
#pragma unroll
        for (int k = 0; k < 8; ++k) sum += v[k];
    }
    // exclusive scan of the quarter sums across q (lanes l, l + 16, l + 32, l + 48)
    uint32_t x = sum;
    uint32_t y = __shfl_up(x, 16);
    if (q >= 1) x += y;
    y = __shfl_up(x, 32);
    if (q >= 2) x += y;
    const uint32_t total = __shfl(x, 48 + l);
    uint32_t run = x - sum;
    for (uint32_t sb = a0; sb < a1; sb += 8) {
        uint32_t v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = sb + k < a1 ? wave_cnt[(size_t)(sb + k) * kBlockTiles + l] : 0u;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            if (sb + k < a1) wave_cnt[(size_t)(sb + k) * kBlockTiles + l] = run;
            run += v[k];
        }
    }
    const int tx = kBlockDim * (b % blocks_x) + (l & 3), ty = kBlockDim * (b / blocks_x) + (l >> 2);
    if (q == 0 && tx < tiles_x && ty < tiles_y) tile_ranges[2 * ((int64_t)ty * tiles_x + tx) + 1] = total;
}

// One workgroup: exclusive scan of the tile lengths in tile order, written as
// [start, end) ranges. Each thread takes kStartsPer consecutive tiles per
// sweep (one sweep covers 8,192 tiles: every image up to 1448 x 1448 tiles of
// 16 pixels in one). Pairs over capacity (the preprocess's count, or the
// lengths' sum) leave every range empty and raise counters[1], which stops the
// emission.
constexpr int kStartsPer = 8;

__global__ __launch_bounds__(kListThreads) void k_tile_starts(int n_tiles, PairCount pairs, uint64_t capacity,
                                                              uint32_t* __restrict__ tile_ranges,
                                                              uint32_t* __restrict__ counters)
{
    __shared__ uint64_t lds16[kListThreads / kWave];
    __shared__ int over;
    if (threadIdx.x == 0) over = pairs.overflow() ? 1 : 0;
    uint64_t carry = 0;   // 64-bit sums: a sum past the capacity is detected, never wrapped
    for (int t0 = 0; t0 < n_tiles; t0 += kListThreads * kStartsPer) {
        const int tb = t0 + (int)threadIdx.x * kStartsPer;
        uint32_t len[kStartsPer];
        uint64_t sum = 0;
#pragma unroll
        for (int k = 0; k < kStartsPer; ++k) {
            len[k] = tb + k < n_tiles ? tile_ranges[2 * (tb + k) + 1] : 0u;
            sum += len[k];
        }
        uint64_t total;
        const uint64_t before = wg_excl_scan_1024(sum, lds16, &total);   // also orders `over`
        uint64_t start = carry + before;
#pragma unroll
        for (int k = 0; k < kStartsPer; ++k) {
            if (tb + k < n_tiles) {
                if (start + len[k] > capacity) over = 1;
                tile_ranges[2 * (tb + k)] = (uint32_t)start;
                tile_ranges[2 * (tb + k) + 1] = (uint32_t)(start + len[k]);
            }
            start += len[k];
        }
        carry += total;
    }
    __syncthreads();
    if (over) {
        for (int t = threadIdx.x; t < n_tiles; t += kListThreads) tile_ranges[2 * t] = tile_ranges[2 * t + 1] = 0u;
    }
    if (threadIdx.x == 0) counters[1] = over ? 1u : 0u;
}

template <bool kTileIds>
__global__ __launch_bounds__(kBlock) void k_tile_emit(const uint32_t* __restrict__ ent_key,
                                                      const uint32_t* __restrict__ ent_gid,
                                                      const uint32_t* __restrict__ block_ranges,
                                                      const uint32_t* __restrict__ seg_base,
                                                      const uint32_t* __restrict__ seg_block,
                                                      const uint32_t* __restrict__ counters, int blocks_x, int tiles_x,
                                                      const uint32_t* __restrict__ wave_off,
                                                      const uint32_t* __restrict__ tile_ranges,
                                                      uint32_t* __restrict__ values, uint32_t* __restrict__ tile_ids)
{
    const uint32_t s = blockIdx.x;
    if (s >= counters[0] || counters[1] != 0u) return;
    const Segment g = segment_of(s, seg_block, seg_base, block_ranges);
    const int bx = (int)(g.b % (uint32_t)blocks_x), by = (int)(g.b / (uint32_t)blocks_x);
    const int lane = __lane_id();
    // lane l: this wave's offset inside the list of tile l
    const uint32_t base_l =
        lane < kBlockTiles ? wave_off[((size_t)s * kSubSegs + (threadIdx.x >> 6)) * kBlockTiles + lane] : 0u;
    uint32_t mask[kSegRounds], gid[kSegRounds];
    load_segment<true>(g, ent_key, ent_gid, mask, gid);
    const uint64_t below = (1ull << lane) - 1ull;
    // tile-major: one running offset live at a time
#pragma unroll
    for (int l = 0; l < kBlockTiles; ++l) {
        const uint32_t tile = (uint32_t)((kBlockDim * by + (l >> 2)) * tiles_x + kBlockDim * bx + (l & 3));
        uint32_t m_any = 0;
#pragma unroll
        for (int r = 0; r < kSegRounds; ++r) m_any |= (mask[r] >> l) & 1u;
        if (__ballot(m_any) == 0) continue;
        // the tile is inside the grid: some entry meets it
        uint32_t off = tile_ranges[2 * tile] + __builtin_amdgcn_readlane(base_l, l);
#pragma unroll
        for (int r = 0; r < kSegRounds; ++r) {
            const bool on = (mask[r] >> l) & 1u;
            const uint64_t m = __ballot(on);
            // inside the tile's range: the counts are those k_tile_count took,
            // and k_tile_starts let no range past the capacity
            if (on) {
                const uint32_t pos = off + (uint32_t)__popcll(m & below);
                values[pos] = gid[r];
                if (kTileIds) tile_ids[pos] = tile;
            }
            off += (uint32_t)__popcll(m);
        }
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

int blocks_x_of(const Cam& cam) { return (cam.tiles_x + kBlockDim - 1) / kBlockDim; }
int blocks_y_of(const Cam& cam) { return (cam.tiles_y + kBlockDim - 1) / kBlockDim; }
int64_t segment_bound(const Cam& cam, uint64_t capacity)
{
    return div_up((int64_t)capacity, kSegEntries) + (int64_t)blocks_x_of(cam) * blocks_y_of(cam);
}

hipError_t launch_entry_offsets(int64_t n, PairCount pairs, const Workspace& ws, hipStream_t s)
{
    const int nb = (int)div_up(n, kDupChunk);
    hipLaunchKernelGGL(k_entry_partial, dim3(nb), dim3(kBlock), 0, s, ws.sorted_rect, n, ws.scan_part);
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kBlock), 0, s, ws.scan_part, nb, pairs, ws.entry_count);
    return hipGetLastError();
}

// Bits of the block id.
static int block_bits(const Cam& cam)
{
    const uint32_t nb = (uint32_t)blocks_x_of(cam) * (uint32_t)blocks_y_of(cam);
    int bits = 0;
    while (bits < 32 && ((nb - 1) >> bits) != 0) ++bits;
    return bits;
}

bool blocks_supported(const Cam& cam) { return block_bits(cam) <= 32 - kMaskBits; }

hipError_t launch_block_entries(const Cam& cam, int64_t n, const uint32_t* order, PairCount entries,
                                const Workspace& ws, hipStream_t s)
{
    const int nb = (int)div_up(n, kDupChunk);
    hipLaunchKernelGGL(k_block_entries, dim3(nb), dim3(kBlock), 0, s, order, ws.sorted_rect, n, ws.scan_part,
                       blocks_x_of(cam), entries, ws.entry_keys_a, ws.entry_vals_a);
    return hipGetLastError();
}

// Stable LSD sort of the entries by block id, the key bits above the tile
// mask (passes of <= 9 bits; none with a single block), then each block's
// entry range (the digit totals of a single pass, else a search of the sorted
// keys) and the segment table.
hipError_t launch_block_sort(const Cam& cam, PairCount entries, const Workspace& ws, BlockEntries* out, hipStream_t s)
{
    const int n_blocks = blocks_x_of(cam) * blocks_y_of(cam);
    const int bits = block_bits(cam);
    const int passes = (bits + kBlockSortBits - 1) / kBlockSortBits;
    uint32_t* kbuf[2] = {ws.entry_keys_a, ws.entry_keys_b};
    uint32_t* vbuf[2] = {ws.entry_vals_a, ws.entry_vals_b};
    int src = 0, shift = kMaskBits;
    // a single pass's digit totals are the blocks' entry counts: its scatter's
    // extra workgroup writes the segment table
    const SegTable seg_one{ws.block_ranges, ws.seg_base, ws.seg_block, ws.list_counters, n_blocks};
    const SegTable seg_none{nullptr, nullptr, nullptr, nullptr, 0};
    for (int p = 0; p < passes; ++p) {
        const int pb = (kMaskBits + bits - shift + (passes - p) - 1) / (passes - p);   // remaining bits spread evenly
        const hipError_t e = block_radix_pass(kbuf[src], vbuf[src], entries, shift, pb, kbuf[src ^ 1],
                                              vbuf[src ^ 1], ws.hist, ws.digit_tot, s,
                                              passes == 1 ? seg_one : seg_none);
        if (e != hipSuccess) return e;
        shift += pb;
        src ^= 1;
    }
    if (passes != 1) {   // none (a single block) or several: ranges by search, then the table
        const dim3 grid((unsigned)div_up(n_blocks + 1, kBlock / kWave));
        hipLaunchKernelGGL(k_ranges, grid, dim3(kBlock), 0, s, kbuf[src], kMaskBits, entries, n_blocks,
                           ws.block_ranges);
        hipLaunchKernelGGL(k_segments, dim3(1), dim3(kListThreads), 0, s, (const uint32_t*)nullptr,
                           ws.block_ranges, n_blocks, ws.seg_base, ws.seg_block, ws.list_counters);
    }
    out->key = kbuf[src];
    out->gid = vbuf[src];
    return hipGetLastError();
}

hipError_t launch_tile_lists(const Cam& cam, PairCount pairs, uint64_t capacity, const Workspace& ws,
                             const BlockEntries& ent, uint32_t* values, uint32_t* tile_ids, uint32_t* tile_ranges,
                             hipStream_t s)
{
    const int bx = blocks_x_of(cam), n_blocks = bx * blocks_y_of(cam);
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const dim3 segs((unsigned)segment_bound(cam, capacity));
    hipLaunchKernelGGL(k_tile_count, segs, dim3(kBlock), 0, s, ent.key, ws.block_ranges, ws.seg_base, ws.seg_block,
                       ws.list_counters, ws.seg_cnt);
    hipLaunchKernelGGL(k_tile_scan, dim3(n_blocks), dim3(kWave), 0, s, ws.seg_base, n_blocks, bx, cam.tiles_x,
                       cam.tiles_y, ws.seg_cnt, tile_ranges);
    hipLaunchKernelGGL(k_tile_starts, dim3(1), dim3(kListThreads), 0, s, n_tiles, pairs, capacity, tile_ranges,
                       ws.list_counters);
    if (tile_ids)
        hipLaunchKernelGGL(k_tile_emit<true>, segs, dim3(kBlock), 0, s, ent.key, ent.gid, ws.block_ranges,
                           ws.seg_base, ws.seg_block, ws.list_counters, bx, cam.tiles_x, ws.seg_cnt, tile_ranges,
                           values, tile_ids);
    else
        hipLaunchKernelGGL(k_tile_emit<false>, segs, dim3(kBlock), 0, s, ent.key, ent.gid, ws.block_ranges,
                           ws.seg_base, ws.seg_block, ws.list_counters, bx, cam.tiles_x, ws.seg_cnt, tile_ranges,
                           values, tile_ids);
    return hipGetLastError();
}

}  // namespace gsr
