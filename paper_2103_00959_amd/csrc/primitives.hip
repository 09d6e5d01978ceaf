// Device-wide building blocks used by the balancer and the CSR -> CSC
// transpose: an exclusive prefix sum and a stable least-significant-digit
// radix sort of (key, value) pairs.  Both are deterministic (integer work,
// fixed tile order); neither allocates.
#include "common.hpp"
#include "internal.hpp"

namespace cogdl {

namespace {

constexpr int kScanBlock = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanBlock * kScanItems;   // 2048

constexpr int kSortBlock = 256;                      // 4 wavefronts
constexpr int kSortItems = 16;
constexpr int kSortTile = kSortBlock * kSortItems;   // 4096
constexpr int kDigits = 256;                         // digits of at most 8 bits
constexpr int kMaxDigitBits = 8;                     // widest digit of a pass

__device__ __forceinline__ int wave_inclusive_scan(int x)
{
    const int lane = lane_id();
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        int y = __builtin_amdgcn_ds_bpermute((lane >= d ? lane - d : lane) << 2, x);
        if (lane >= d) x += y;
    }
    return x;
}

// Exclusive scan of one value per thread across a 256-thread block; returns
// the exclusive prefix and writes the block total to *total.
__device__ __forceinline__ int block_exclusive_scan(int x, int *total)
{
    __shared__ int wsum[kScanBlock / kWave];
    const int lane = lane_id(), w = threadIdx.x / kWave;
    int inc = wave_inclusive_scan(x);
    if (lane == kWave - 1) wsum[w] = inc;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kScanBlock / kWave; ++i) {
        if (i < w) before += wsum[i];
        all += wsum[i];
    }
    __syncthreads();
    *total = all;
    return before + inc - x;
}

// K arrays scanned side by side (one launch for all of them); sums of the
// tiles of array k at tile_sums[k * stride + tile].
template <int K>
struct ScanSet {
    const int32_t *in[K];
    int32_t *out[K];
};

template <int K>
__global__ __launch_bounds__(kScanBlock) void k_tile_reduce(ScanSet<K> a, int64_t n,
                                                            int32_t *__restrict__ tile_sums,
                                                            int64_t stride)
{
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        int s = 0;
#pragma unroll
        for (int i = 0; i < kScanItems; ++i)
            if (base + i < n) s += a.in[k][base + i];
        int total;
        block_exclusive_scan(s, &total);
        if (threadIdx.x == 0) tile_sums[k * stride + blockIdx.x] = total;
    }
}

// Scan one tile of each array and add the tile's offset: tile_offs[k * stride +
// tile] when given; else, with `sums` given, the sum of sums[k * stride + t]
// over the tiles t before this one (added up by the block itself, so a scan
// of up to kDirectTiles tiles needs no second level); else 0 (single tile).
// The block holding the last element also writes out[n] = total.
constexpr int64_t kDirectTiles = 8192;

template <int K>
__global__ __launch_bounds__(kScanBlock) void k_tile_scan(ScanSet<K> a, int64_t n,
                                                          const int32_t *__restrict__ tile_offs,
                                                          int64_t stride,
                                                          const int32_t *__restrict__ sums)
{
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        int before = 0;
        if (!tile_offs && sums) {
            int part = 0;
            for (int t = threadIdx.x; t < (int)blockIdx.x; t += kScanBlock) part += sums[k * stride + t];
            int all;
            block_exclusive_scan(part, &all);
            before = all;
        }
        int v[kScanItems];
        int s = 0;
#pragma unroll
        for (int i = 0; i < kScanItems; ++i) {
            v[i] = (base + i < n) ? a.in[k][base + i] : 0;
            s += v[i];
        }
        int total;
        int run = block_exclusive_scan(s, &total);   // contains a barrier: all reads done
        const int off = tile_offs ? tile_offs[k * stride + blockIdx.x] : before;
        run += off;
#pragma unroll
        for (int i = 0; i < kScanItems; ++i) {
            if (base + i < n) a.out[k][base + i] = run;
            run += v[i];
        }
        if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) a.out[k][n] = off + total;
    }
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// Per-tile histogram of one digit (bits [shift, shift + dbits) of the key),
// stored digit-major so that an exclusive scan of the whole table yields every
// (digit, tile) start slot.  Each wavefront counts into kHistCopies LDS copies
// (lane % kHistCopies picks one), so the lanes of a wavefront that share a
// digit, common on the high digits of power-law keys, collide on one LDS
// address a quarter as often.
constexpr int kHistCopies = 4;

__global__ __launch_bounds__(kSortBlock) void k_radix_hist(const uint32_t *__restrict__ keys, int64_t n,
                                                           int shift, int dbits, int n_tiles,
                                                           int32_t *__restrict__ hist,
                                                           const int32_t *__restrict__ rowptr,
                                                           int64_t n_rows,
                                                           int32_t *__restrict__ start_rows)
{
    constexpr int kCopies = (kSortBlock / kWave) * kHistCopies;
    __shared__ int32_t h[kCopies][kDigits];
#pragma unroll
    for (int w = 0; w < kCopies; ++w) h[w][threadIdx.x] = 0;
    __syncthreads();
    const int copy = (threadIdx.x / kWave) * kHistCopies + lane_id() % kHistCopies;
    const uint32_t mask = (1u << dbits) - 1u;
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    uint32_t key[kSortItems];
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        const int64_t e = base + (int64_t)i * kSortBlock + threadIdx.x;
        key[i] = keys[e < n ? e : n - 1];
    }
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        const int64_t e = base + (int64_t)i * kSortBlock + threadIdx.x;
        if (e < n) atomicAdd(&h[copy][(key[i] >> shift) & mask], 1);
    }
    __syncthreads();
    if (threadIdx.x < (1 << dbits)) {
        int c = 0;
#pragma unroll
        for (int w = 0; w < kCopies; ++w) c += h[w][threadIdx.x];
        hist[(int64_t)threadIdx.x * n_tiles + blockIdx.x] = c;
    }
    // the scatter's CSR rows: the row holding the first element of each
    // wavefront's quarter of the tile, found here where latency is cheap
    if (start_rows) {
        const int64_t wb = base + (int64_t)(threadIdx.x / kWave) * kWave * kSortItems;
        if (wb < n) {
            const int64_t r = RowCursor::find(rowptr, n_rows, wb);
            if (lane_id() == 0) start_rows[(int64_t)blockIdx.x * (kSortBlock / kWave) + threadIdx.x / kWave] = (int32_t)r;
        }
    }
}

// Tile handled by workgroup b of nb.  Workgroups are dealt to the 8 XCDs
// round-robin (b % 8), so XCD x gets the contiguous tile range
// [x * nb / 8, (x + 1) * nb / 8) instead of every 8th tile: the tiles running
// together on one XCD then write adjacent pieces of each digit's output run,
// and the cache lines split between two tiles are completed in that XCD's L2
// before they go to HBM.  Any bijection is correct; this one is a speed choice.
__device__ __forceinline__ int xcd_tile(int b, int nb)
{
    constexpr int kXcds = 8;
    const int x = b % kXcds, per = nb / kXcds, rem = nb % kXcds;
    return x * per + (x < rem ? x : rem) + b / kXcds;
}

// Stable scatter of one tile.  Wavefront w owns the contiguous quarter
// [w * 1024, (w + 1) * 1024) of the tile and walks it 64 keys at a time; the
// rank of a key among equal digits is the number of lower lanes with the same
// digit (found with one ballot per digit bit) plus the running per-wave count.  All
// arrays of the tile are loaded up front (one memory round trip), then staged
// in LDS in tile-sorted order two at a time and written out by consecutive
// threads, so equal digits leave as contiguous runs instead of scattered
// 4-byte stores.  NP extra 32-bit payloads travel with each key; ROWS: the
// first payload is the CSR row of each element, resolved by each wavefront
// for its 16 chunks of 64 consecutive elements with a RowCursor started at
// the row k_radix_hist found for that wavefront (start_rows).
template <int NP, bool ROWS>
__global__ __launch_bounds__(kSortBlock) void k_radix_scatter(
    const uint32_t *__restrict__ keys_in, const uint32_t *__restrict__ vals_in,
    uint32_t *__restrict__ keys_out, uint32_t *__restrict__ vals_out, int64_t n, int shift,
    int dbits, int n_tiles, const int32_t *__restrict__ offsets, RadixPayload p0, RadixPayload p1,
    const int32_t *__restrict__ start_rows)
{
    constexpr int kWaves = kSortBlock / kWave;
    __shared__ int32_t wcnt[kWaves][kDigits];   // per-wave counts, then tile-local run starts
    __shared__ int32_t dstart[kDigits];         // tile-local start of each digit
    __shared__ int32_t gstart[kDigits];         // global start of this tile's run of each digit
    __shared__ uint32_t stage[2][kSortTile];
    __shared__ uint8_t qdig[kSortTile];
    const int tid = threadIdx.x, w = tid / kWave, lane = lane_id();
    const uint32_t dmask = (1u << dbits) - 1u;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) wcnt[i][tid] = 0;

    const int tile = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t tile0 = (int64_t)tile * kSortTile;
    const int count = (int)((n - tile0) < kSortTile ? (n - tile0) : kSortTile);
    const int64_t base = tile0 + (int64_t)w * kWave * kSortItems;
    uint32_t key[kSortItems], val[kSortItems], pa[NP > 0 ? kSortItems : 1], pb[NP > 1 ? kSortItems : 1];
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        const int64_t e = base + i * kWave + lane;
        const int64_t ec = e < n ? e : n - 1;     // clamped: loads need no branch
        key[i] = keys_in[ec];
        val[i] = vals_in ? vals_in[ec] : (uint32_t)e;
        if constexpr (NP > 0 && !ROWS) pa[i] = p0.in[ec];
        if constexpr (NP > 1) pb[i] = p1.in[ec];
    }
    if constexpr (ROWS) {
        static_assert(NP > 0 && kSortItems % 4 == 0, "rows need a payload slot");
        if (base < n) {                               // uniform across the wavefront
            RowCursor rc;
            rc.start_at(p0.rowptr, p0.n_rows, start_rows[(int64_t)tile * kWaves + w]);
#pragma unroll
            for (int i0 = 0; i0 < kSortItems; i0 += 4) {
                int64_t e[4], row[4];
                bool want[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    e[j] = base + (int64_t)(i0 + j) * kWave + lane;
                    want[j] = e[j] < n;
                }
                rc.resolve<4>(e, want, row);
#pragma unroll
                for (int j = 0; j < 4; ++j) pa[i0 + j] = (uint32_t)row[j];
            }
        }
    }
    __syncthreads();

    const uint64_t lower = __lanemask_lt();
    int local[kSortItems];
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        const bool valid = base + i * kWave + lane < n;
        const int d = (int)((key[i] >> shift) & dmask);
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < kMaxDigitBits; ++b) {
            if (b >= dbits) break;
            const int bit = (d >> b) & 1;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const int rank = __popcll(peers & lower);
        int old = 0;
        if (valid) old = wcnt[w][d];
        local[i] = valid ? old + rank : -1;
        if (valid && rank == 0) wcnt[w][d] = old + __popcll(peers);
    }
    __syncthreads();
    {
        // tile-local start of digit `tid`, and of each wave's share of it
        int tot = 0;
#pragma unroll
        for (int i = 0; i < kWaves; ++i) tot += wcnt[i][tid];
        int all;
        const int start = block_exclusive_scan(tot, &all);
        dstart[tid] = start;
        gstart[tid] = tid <= (int)dmask ? offsets[(int64_t)tid * n_tiles + tile] : 0;
        int run = start;
#pragma unroll
        for (int i = 0; i < kWaves; ++i) {
            const int c = wcnt[i][tid];
            wcnt[i][tid] = run;
            run += c;
        }
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kSortItems; ++i) {
        if (local[i] >= 0) {
            const int d = (int)((key[i] >> shift) & dmask);
            local[i] += wcnt[w][d];
            stage[0][local[i]] = key[i];
            stage[1][local[i]] = val[i];
            qdig[local[i]] = (uint8_t)d;
        }
    }
    __syncthreads();
    for (int q = tid; q < count; q += kSortBlock) {
        const int d = qdig[q];
        const int pos = gstart[d] + (q - dstart[d]);
        if (keys_out) keys_out[pos] = stage[0][q];
        vals_out[pos] = stage[1][q];
    }
    if constexpr (NP > 0) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kSortItems; ++i) {
            if (local[i] >= 0) {
                stage[0][local[i]] = pa[i];
                if constexpr (NP > 1) stage[1][local[i]] = pb[i];
            }
        }
        __syncthreads();
        for (int q = tid; q < count; q += kSortBlock) {
            const int d = qdig[q];
            const int pos = gstart[d] + (q - dstart[d]);
            p0.out[pos] = stage[0][q];
            if constexpr (NP > 1) p1.out[pos] = stage[1][q];
        }
    }
}

int64_t scan_levels_ints(int64_t n)
{
    int64_t total = 0;
    while (n > kScanTile) {
        int64_t t = (n + kScanTile - 1) / kScanTile;
        total += t + 1;
        n = t;
    }
    return total;
}

template <int K>
hipError_t scan_rec(ScanSet<K> a, int64_t n, int32_t *ws, hipStream_t s)
{
    if (n <= 0) {
        for (int k = 0; k < K; ++k) COGDL_LAUNCH_HIP("fill", k_fill_i32, 1, 64, s, a.out[k], 1, 0);
        return hipSuccess;
    }
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    if (tiles == 1) {
        COGDL_LAUNCH_HIP("scan_tile", k_tile_scan<K>, 1, kScanBlock, s, a, n, nullptr, 0, nullptr);
        return hipSuccess;
    }
    // the tile sums of array k at ws[k * (tiles + 1)], scanned in place
    const int64_t stride = tiles + 1;
    int32_t *sums = ws;
    COGDL_LAUNCH_HIP("scan_reduce", k_tile_reduce<K>, (unsigned)tiles, kScanBlock, s, a, n, sums,
                     stride);
    if (tiles <= kDirectTiles) {
        COGDL_LAUNCH_HIP("scan_tile", k_tile_scan<K>, (unsigned)tiles, kScanBlock, s, a, n, nullptr,
                         stride, sums);
        return hipSuccess;
    }
    ScanSet<K> b;
    for (int k = 0; k < K; ++k) {
        b.in[k] = sums + k * stride;
        b.out[k] = sums + k * stride;
    }
    hipError_t e = scan_rec<K>(b, tiles, ws + K * stride, s);
    if (e != hipSuccess) return e;
    COGDL_LAUNCH_HIP("scan_tile", k_tile_scan<K>, (unsigned)tiles, kScanBlock, s, a, n, sums, stride,
                     nullptr);
    return hipSuccess;
}

}  // namespace

size_t scan_workspace_bytes(int64_t n, int arrays)
{
    return (size_t)(arrays * scan_levels_ints(n) + 16) * 4;
}

hipError_t exclusive_scan(const int32_t *in, int32_t *out, int64_t n, void *ws, hipStream_t s)
{
    ScanSet<1> a;
    a.in[0] = in;
    a.out[0] = out;
    return scan_rec<1>(a, n, static_cast<int32_t *>(ws), s);
}

hipError_t exclusive_scan3(int32_t *a0, int32_t *a1, int32_t *a2, int64_t n, void *ws, hipStream_t s)
{
    ScanSet<3> a;
    a.in[0] = a.out[0] = a0;
    a.in[1] = a.out[1] = a1;
    a.in[2] = a.out[2] = a2;
    return scan_rec<3>(a, n, static_cast<int32_t *>(ws), s);
}

hipError_t fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s)
{
    if (n <= 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    COGDL_LAUNCH_HIP("fill", k_fill_i32, (unsigned)blocks, 256, s, p, n, v);
    return hipSuccess;
}

// Workspace of a radix sort of n keys: the digit table (+ its scan's scratch)
// and one start row per wavefront of a tile (rows generated from rowptr).
size_t radix_workspace_bytes(int64_t n)
{
    const int64_t tiles = (n + kSortTile - 1) / kSortTile;
    const int64_t hist = (int64_t)kDigits * (tiles > 0 ? tiles : 1) + 1;
    size_t b = (size_t)(hist + 64) * 4;
    b = (b + 255) & ~size_t(255);
    b += (scan_workspace_bytes(hist) + 255) & ~size_t(255);
    return b + (size_t)(tiles > 0 ? tiles : 1) * (kSortBlock / kWave) * 4;
}

hipError_t radix_sort_pairs(const uint32_t *keys_in, const uint32_t *vals_in, uint32_t *keys_out,
                            uint32_t *vals_out, int64_t n, int bits, uint32_t *ping_keys,
                            uint32_t *ping_vals, void *ws, hipStream_t s, RadixPayload pay0,
                            RadixPayload pay1)
{
    if (n <= 0) return hipSuccess;
    const int np = (pay0.in || pay0.rowptr) ? (pay1.in ? 2 : 1) : 0;
    const int64_t tiles = (n + kSortTile - 1) / kSortTile;
    const int64_t hist_n = (int64_t)kDigits * tiles;
    int32_t *hist = static_cast<int32_t *>(ws);
    size_t hist_bytes = ((size_t)(hist_n + 1 + 64) * 4 + 255) & ~size_t(255);
    void *scan_ws = static_cast<char *>(ws) + hist_bytes;
    int32_t *start_rows = reinterpret_cast<int32_t *>(
        static_cast<char *>(scan_ws) + ((scan_workspace_bytes(hist_n + 1) + 255) & ~size_t(255)));

    // as few passes as digits of at most 8 bits allow, the bits spread evenly
    // over them (longer runs per digit than a short last pass gives), a
    // remainder going to the last passes: a narrower digit gives longer runs,
    // which matters most in the first pass (it also generates the CSR rows)
    // and least in the last (the high bits of power-law keys take few values)
    int passes = (bits + kMaxDigitBits - 1) / kMaxDigitBits;
    if (passes < 1) passes = 1;
    const uint32_t *src_k = keys_in;
    const uint32_t *src_v = vals_in;
    RadixPayload a = pay0, b = pay1;
    int shift = 0;
    for (int p = 0; p < passes; ++p) {
        const bool last = (p == passes - 1);
        int dbits = (bits - shift) / (passes - p);
        if (dbits < 1) dbits = 1;
        uint32_t *dst_k = last ? keys_out : ping_keys + (p & 1) * n;
        uint32_t *dst_v = last ? vals_out : ping_vals + (p & 1) * n;
        RadixPayload pa{a.in, last ? pay0.out : (pay0.ping ? pay0.ping + (p & 1) * n : nullptr), nullptr};
        const bool rows = p == 0 && pay0.rowptr != nullptr && pay0.in == nullptr;
        pa.rowptr = pay0.rowptr;
        pa.n_rows = pay0.n_rows;
        RadixPayload pb{b.in, last ? pay1.out : (pay1.ping ? pay1.ping + (p & 1) * n : nullptr), nullptr};
        const int64_t used = (int64_t)(1 << dbits) * tiles;
        COGDL_LAUNCH_HIP("radix_hist", k_radix_hist, (unsigned)tiles, kSortBlock, s, src_k, n, shift,
                         dbits, (int)tiles, hist, pay0.rowptr, pay0.n_rows, rows ? start_rows : nullptr);
        hipError_t e = exclusive_scan(hist, hist, used, scan_ws, s);
        if (e != hipSuccess) return e;
#define COGDL_SCATTER(NPV, ROWSV)                                                                \
    COGDL_LAUNCH_HIP("radix_scatter", (k_radix_scatter<NPV, ROWSV>), (unsigned)tiles, kSortBlock, s, \
                     src_k, src_v, dst_k, dst_v, n, shift, dbits, (int)tiles, hist, pa, pb,          \
                     start_rows)
        if (np == 0) COGDL_SCATTER(0, false);
        else if (np == 1 && rows) COGDL_SCATTER(1, true);
        else if (np == 1) COGDL_SCATTER(1, false);
        else if (rows) COGDL_SCATTER(2, true);
        else COGDL_SCATTER(2, false);
#undef COGDL_SCATTER
        src_k = dst_k;
        src_v = dst_v;
        a.in = pa.out;
        b.in = pb.out;
        shift += dbits;
    }
    return hipSuccess;
}

RowMap row_map(int64_t width, int elem_bytes, int unit_elems, bool aligned16)
{
    RowMap m;
    const int v16 = 16 / elem_bytes;
    m.vec = (aligned16 && width % v16 == 0 && unit_elems % v16 == 0) ? v16 : 1;
    const int64_t lanes = (width + m.vec - 1) / m.vec;
    if (lanes <= kWave) {
        m.S = next_pow2((int)(lanes > 0 ? lanes : 1));
        m.ch = 1;
    } else {
        m.S = kWave;
        const int64_t ch = (lanes + kWave - 1) / kWave;
        m.ch = ch <= 1 ? 1 : (ch <= 2 ? 2 : 4);
    }
    m.log2S = log2i(m.S);
    m.slab = m.S * m.ch * m.vec;
    m.n_slabs = (int)((width + m.slab - 1) / m.slab);
    if (m.n_slabs < 1) m.n_slabs = 1;
    return m;
}

}  // namespace cogdl
