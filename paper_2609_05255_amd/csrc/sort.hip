// Depth-sorted per-tile lists (Sec. 3.1 "depth-sorted order"): the pairs must
// come out ordered by (tile, depth key, Gaussian index).
//
// Instead of radix-sorting P 45-bit (tile, depth) keys, the Gaussians are
// sorted once by depth (4 stable 8-bit LSD passes over n 32-bit keys with the
// index as value, so equal depths stay in index order), the pairs are emitted
// in that order, and a stable LSD sort on the tile id alone (ceil(log2 T)/8
// passes) finishes the job: stability keeps (depth, index) order within a tile.
//
// One radix pass = k_radix_hist (per-workgroup digit counts) + k_radix_scan
// (exclusive offsets per digit over workgroups) + k_radix_scatter (stable
// rank inside the workgroup with wave64 ballots, then scatter).
#include "gs_internal.h"

namespace gsr {

namespace {

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

// Lanes of this wave holding the same 8-bit digit (restricted to valid lanes).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid)
{
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        const bool bit = (d >> b) & 1u;
        const uint64_t bm = __ballot(bit);
        m &= bit ? bm : ~bm;
    }
    return m;
}

__global__ __launch_bounds__(kBlock) void k_radix_hist(const uint32_t* __restrict__ keys, uint64_t count, int shift,
                                                       uint32_t* __restrict__ hist, int nblocks)
{
    __shared__ uint32_t h[4][kRadix];
    for (int k = threadIdx.x; k < 4 * kRadix; k += kBlock) (&h[0][0])[k] = 0;
    __syncthreads();
    const int wave = threadIdx.x >> 6;
    const uint64_t base = (uint64_t)blockIdx.x * kSortTile;
#pragma unroll 4
    for (int r = 0; r < kSortItems; ++r) {
        const uint64_t idx = base + (uint64_t)r * kBlock + threadIdx.x;
        if (idx < count) atomicAdd(&h[wave][(keys[idx] >> shift) & 0xFFu], 1u);
    }
    __syncthreads();
    const int d = threadIdx.x;
    hist[(size_t)d * nblocks + blockIdx.x] = h[0][d] + h[1][d] + h[2][d] + h[3][d];
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

__global__ __launch_bounds__(kBlock) void k_radix_scatter(const uint32_t* __restrict__ keys_in,
                                                          const uint32_t* __restrict__ vals_in, uint64_t count,
                                                          int shift, const uint32_t* __restrict__ hist, int nblocks,
                                                          const uint32_t* __restrict__ digit_tot,
                                                          uint32_t* __restrict__ keys_out,
                                                          uint32_t* __restrict__ vals_out)
{
    __shared__ uint32_t run[kRadix];
    __shared__ uint32_t cnt[4][kRadix];
    __shared__ uint32_t lds4[4];
    const int t = threadIdx.x, wave = t >> 6;
    const uint32_t base_d = block_excl_scan(digit_tot[t], lds4, nullptr);
    run[t] = base_d + hist[(size_t)t * nblocks + blockIdx.x];
    for (int w = 0; w < 4; ++w) cnt[w][t] = 0;
    __syncthreads();
    const uint64_t base = (uint64_t)blockIdx.x * kSortTile;
    for (int r = 0; r < kSortItems; ++r) {
        const uint64_t idx = base + (uint64_t)r * kBlock + t;
        const bool valid = idx < count;
        uint32_t key = 0, val = 0;
        if (valid) {
            key = keys_in[idx];
            val = vals_in ? vals_in[idx] : (uint32_t)idx;
        }
        const uint32_t d = (key >> shift) & 0xFFu;
        const uint64_t peers = match_digit(d, valid);
        const uint32_t rank = (uint32_t)__popcll(peers & lanemask_lt());
        if (valid && rank == 0) cnt[wave][d] = (uint32_t)__popcll(peers);
        __syncthreads();
        if (valid) {
            uint32_t pos = run[d] + rank;
            for (int w = 0; w < wave; ++w) pos += cnt[w][d];
            keys_out[pos] = key;
            vals_out[pos] = val;
        }
        __syncthreads();
        run[t] += cnt[0][t] + cnt[1][t] + cnt[2][t] + cnt[3][t];
        cnt[0][t] = cnt[1][t] = cnt[2][t] = cnt[3][t] = 0;
        __syncthreads();
    }
}

// One stable LSD pass; vals_in == nullptr means value = position.
hipError_t radix_pass(const uint32_t* keys_in, const uint32_t* vals_in, uint64_t count, int shift,
                      uint32_t* keys_out, uint32_t* vals_out, uint32_t* hist, uint32_t* digit_tot, hipStream_t s)
{
    const int nblocks = (int)div_up((int64_t)count, kSortTile);
    hipLaunchKernelGGL(k_radix_hist, dim3(nblocks), dim3(kBlock), 0, s, keys_in, count, shift, hist, nblocks);
    hipLaunchKernelGGL(k_radix_scan, dim3(kRadix), dim3(kBlock), 0, s, hist, nblocks, digit_tot);
    hipLaunchKernelGGL(k_radix_scatter, dim3(nblocks), dim3(kBlock), 0, s, keys_in, vals_in, count, shift, hist,
                       nblocks, digit_tot, keys_out, vals_out);
    return hipGetLastError();
}

// ---- pair offsets in depth order and pair emission ---------------------------

__global__ __launch_bounds__(kBlock) void k_pair_partial(const uint32_t* __restrict__ order,
                                                         const uint32_t* __restrict__ tiles_touched, int64_t n,
                                                         uint32_t* __restrict__ part)
{
    __shared__ uint32_t lds4[4];
    const int64_t base = (int64_t)blockIdx.x * kSortTile + (int64_t)threadIdx.x * kSortItems;
    uint32_t sum = 0;
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + k;
        if (i < n) sum += tiles_touched[order[i]];
    }
    uint32_t total;
    block_excl_scan(sum, lds4, &total);
    if (threadIdx.x == 0) part[blockIdx.x] = total;
}

// Exclusive scan of the per-workgroup totals (one workgroup).
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

// Emits the (tile, Gaussian) pairs of the depth-ordered Gaussians; each
// Gaussian's tiles in row-major order of its rectangle.
__global__ __launch_bounds__(kBlock) void k_duplicate(const uint32_t* __restrict__ order,
                                                      const uint32_t* __restrict__ tiles_touched,
                                                      const gs_splat* __restrict__ splats, int64_t n,
                                                      const uint32_t* __restrict__ part, int tiles_x,
                                                      uint32_t capacity, uint32_t* __restrict__ keys,
                                                      uint32_t* __restrict__ vals)
{
    __shared__ uint32_t lds4[4];
    const int64_t base = (int64_t)blockIdx.x * kSortTile + (int64_t)threadIdx.x * kSortItems;
    uint32_t sum = 0;
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + k;
        if (i < n) sum += tiles_touched[order[i]];
    }
    uint32_t off = part[blockIdx.x] + block_excl_scan(sum, lds4, nullptr);
    for (int k = 0; k < kSortItems; ++k) {
        const int64_t i = base + k;
        if (i >= n) break;
        const uint32_t g = order[i];
        if (tiles_touched[g] == 0) continue;
        const float2 rr = *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(splats + g) + 10);
        const uint32_t r01 = __float_as_uint(rr.x), r23 = __float_as_uint(rr.y);
        const int x0 = (int)(r01 & 0xFFFF), y0 = (int)(r01 >> 16);
        const int x1 = (int)(r23 & 0xFFFF), y1 = (int)(r23 >> 16);
        for (int ty = y0; ty < y1; ++ty)
            for (int tx = x0; tx < x1; ++tx) {
                if (off < capacity) {   // only a num_pairs that disagrees with the preprocess gets here
                    keys[off] = (uint32_t)(ty * tiles_x + tx);
                    vals[off] = g;
                }
                ++off;
            }
    }
}

__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* a, uint32_t count, uint32_t v)
{
    uint32_t lo = 0, hi = count;
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if (a[mid] < v) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kBlock) void k_ranges(const uint32_t* __restrict__ sorted_tiles, uint32_t count,
                                                   int n_tiles, uint32_t* __restrict__ ranges)
{
    const int t = blockIdx.x * kBlock + threadIdx.x;
    if (t >= n_tiles) return;
    ranges[2 * t] = lower_bound_u32(sorted_tiles, count, (uint32_t)t);
    ranges[2 * t + 1] = lower_bound_u32(sorted_tiles, count, (uint32_t)t + 1);
}

}  // namespace

hipError_t launch_depth_sort(int64_t n, const uint32_t* depth_key, const Workspace& ws, const uint32_t** order_out,
                             hipStream_t s)
{
    const uint32_t* kin = depth_key;
    const uint32_t* vin = nullptr;
    uint32_t* kbuf[2] = {ws.keys_a, ws.keys_b};
    uint32_t* vbuf[2] = {ws.vals_a, ws.vals_b};
    for (int p = 0; p < 4; ++p) {
        hipError_t e = radix_pass(kin, vin, (uint64_t)n, 8 * p, kbuf[p & 1], vbuf[p & 1], ws.hist,
                                  ws.digit_tot + kRadix * p, s);
        if (e != hipSuccess) return e;
        kin = kbuf[p & 1];
        vin = vbuf[p & 1];
    }
    *order_out = vin;
    return hipSuccess;
}

hipError_t launch_pair_offsets(int64_t n, const uint32_t* order, const uint32_t* tiles_touched, const Workspace& ws,
                               hipStream_t s)
{
    const int nb = (int)div_up(n, kSortTile);
    hipLaunchKernelGGL(k_pair_partial, dim3(nb), dim3(kBlock), 0, s, order, tiles_touched, n, ws.scan_part);
    hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kBlock), 0, s, ws.scan_part, nb);
    return hipGetLastError();
}

hipError_t launch_duplicate(const Cam& cam, int64_t n, const uint32_t* order, const gs_preprocessed& pre,
                            const Workspace& ws, uint32_t capacity, uint32_t* keys_out, uint32_t* vals_out,
                            hipStream_t s)
{
    const int nb = (int)div_up(n, kSortTile);
    hipLaunchKernelGGL(k_duplicate, dim3(nb), dim3(kBlock), 0, s, order, pre.tiles_touched, pre.splats, n,
                       ws.scan_part, cam.tiles_x, capacity, keys_out, vals_out);
    return hipGetLastError();
}

int tile_sort_passes(const Cam& cam)
{
    const uint32_t n_tiles = (uint32_t)cam.tiles_x * (uint32_t)cam.tiles_y;
    int bits = 0;
    while (bits < 32 && ((n_tiles - 1) >> bits) != 0) ++bits;
    return (bits + 7) / 8;
}

hipError_t launch_tile_sort(const Cam& cam, uint64_t num_pairs, const Workspace& ws, uint32_t* values,
                            uint32_t* tile_ids_out, const uint32_t** sorted_tiles, hipStream_t s)
{
    const int passes = tile_sort_passes(cam);
    uint32_t* kbuf[2] = {ws.pair_keys_a, ws.pair_keys_b};
    uint32_t* vbuf[2] = {ws.pair_vals_a, ws.pair_vals_b};
    int src = 0;
    for (int p = 0; p < passes; ++p) {
        const bool last = p == passes - 1;
        uint32_t* kout = last ? (tile_ids_out ? tile_ids_out : kbuf[src ^ 1]) : kbuf[src ^ 1];
        uint32_t* vout = last ? values : vbuf[src ^ 1];
        hipError_t e = radix_pass(kbuf[src], vbuf[src], num_pairs, 8 * p, kout, vout, ws.hist, ws.digit_tot, s);
        if (e != hipSuccess) return e;
        if (last) *sorted_tiles = kout;
        src ^= 1;
    }
    return hipSuccess;
}

hipError_t launch_ranges(const Cam& cam, uint64_t num_pairs, const uint32_t* sorted_tiles, uint32_t* tile_ranges,
                         hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_ranges, dim3((unsigned)div_up(n_tiles, kBlock)), dim3(kBlock), 0, s, sorted_tiles,
                       (uint32_t)num_pairs, n_tiles, tile_ranges);
    return hipGetLastError();
}

}  // namespace gsr
