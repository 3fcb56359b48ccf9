// Stable LSD radix sort of (uint64 key, uint32 value) pairs and the
// schedule output pass (canonical order, caller chunk ids, reductions).
#include "pccl_internal.h"

namespace pccl {
namespace {

constexpr uint32_t SORT_PER = SORT_TILE / SORT_THREADS;  // elements of a tile per thread

// A pass with tgate >= 0 sorts a byte of the start time and runs only if the
// collective time has bits at or above tgate (start times are below it), so
// the number of time bytes follows the device's collective time without a
// host round trip.  tgate < 0: the pass always runs.
__device__ inline bool pass_active(const Layout &ly, int tgate)
{
    return tgate < 0 || (ly.ctl->cstar >> tgate) != 0u;
}

// The send log is complete: the output kernels, which index tables by the
// logged values, run only then (otherwise the call reports an error).
__device__ inline bool log_complete(const Layout &ly)
{
    return !ly.ctl->error && !ly.ctl->abort && ly.ctl->n_log == ly.ctl->needs_total;
}

// Buffer holding the order before pass `pass` of a sort.  Pass 0 takes it
// from sort_cur (buffer 0 after a reset); later passes from sort_buf, which
// each pass's scatter writes for the next one, so no kernel rewrites a
// field the blocks of the same kernel read.
__device__ inline uint32_t pass_src(const Layout &ly, uint32_t pass, bool reset)
{
    return pass ? ly.ctl->sort_buf[pass] : (reset ? 0u : ly.ctl->sort_cur);
}

// Per-tile digit histogram, stored digit-major with 16-bit counts (a tile
// holds at most 4,096 of a digit), hist16[digit * stride + tile] (stride =
// hist_stride(tiles); the last tile zeroes the row's padding), for
// scatters that read a digit's row, or tile-major with 32-bit counts,
// hist[tile * 256 + digit], for the scan kernel (coalesced over digits).  A thread's keys are loaded together (indices past n reread the
// last key and are not counted), so the tile costs one memory round trip.
// Pass 0 also records the sort's start buffer.
template <bool DIGIT_MAJOR>
__global__ void __launch_bounds__(SORT_THREADS) k_hist(Layout ly, uint64_t n, int shift, uint32_t tiles, int tgate,
                                                       uint32_t pass, bool reset)
{
    const uint32_t tid = threadIdx.x, tile = blockIdx.x;
    const uint32_t src = pass_src(ly, pass, reset);
    if (pass == 0 && tile == 0 && tid == 0) ly.ctl->sort_buf[0] = src;
    if (!pass_active(ly, tgate)) return;
    __shared__ uint32_t cnt[256];
    cnt[tid] = 0;
    __syncthreads();
    const uint64_t *key = ly.skey[src];
    const uint64_t base = (uint64_t)tile * SORT_TILE;
    uint32_t dg[SORT_PER];
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++)
        dg[u] = (uint32_t)(key[min(base + u * SORT_THREADS + tid, n - 1)] >> shift) & 255u;
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++)
        if (base + u * SORT_THREADS + tid < n) atomicAdd(&cnt[dg[u]], 1u);
    __syncthreads();
    if (DIGIT_MAJOR) {
        uint16_t *row = reinterpret_cast<uint16_t *>(ly.hist) + (uint64_t)tid * hist_stride(tiles);
        row[tile] = (uint16_t)cnt[tid];
        if (tile == tiles - 1)
            for (uint32_t t = tiles; t < hist_stride(tiles); t++) row[t] = 0;
    } else {
        ly.hist[(uint64_t)tile * 256 + tid] = cnt[tid];
    }
}

// Sorts of more than OWN_PREFIX_TILES tiles scan the histogram in a kernel
// of its own (one workgroup) instead of every tile reading its digit's whole
// row, which grows with the square of the tile count.
constexpr uint32_t OWN_PREFIX_TILES = 256;
constexpr uint32_t SCAN_SPLIT = 4;

// Exclusive scan of the tile-major histogram in (digit, tile) order, in
// place, and the skip decision (some digit holds every element).  Four
// threads per digit each take a quarter of the tiles, so a thread has few
// dependent loads to wait for; a wave's loads cover 64 adjacent digits.
__global__ void __launch_bounds__(256 * SCAN_SPLIT) k_scan(Layout ly, uint64_t n, uint32_t tiles, int tgate)
{
    if (!pass_active(ly, tgate)) return;
    __shared__ uint32_t part[SCAN_SPLIT][256];
    __shared__ uint32_t pre[256];
    const uint32_t d = threadIdx.x & 255u, q = threadIdx.x >> 8;
    const uint32_t per = (tiles + SCAN_SPLIT - 1) / SCAN_SPLIT;
    const uint32_t t0 = min(q * per, tiles), t1 = min(t0 + per, tiles);
    uint32_t tot = 0;
#pragma unroll 16
    for (uint32_t t = t0; t < t1; t++) tot += ly.hist[(uint64_t)t * 256 + d];
    part[q][d] = tot;
    __syncthreads();
    uint32_t all = 0;
    for (uint32_t r = 0; r < SCAN_SPLIT; r++) all += part[r][d];
    if (q == 0) pre[d] = all;
    const bool skip = __syncthreads_or(all == (uint32_t)n);
    if (threadIdx.x == 0) ly.ctl->sort_skip = skip;
    if (skip) return;
    for (uint32_t off = 1; off < 256; off <<= 1) {
        const uint32_t v = (q == 0 && d >= off) ? pre[d - off] : 0u;
        __syncthreads();
        if (q == 0) pre[d] += v;
        __syncthreads();
    }
    uint32_t run = pre[d] - all;  // exclusive prefix over digits
    for (uint32_t r = 0; r < q; r++) run += part[r][d];
#pragma unroll 16
    for (uint32_t t = t0; t < t1; t++) {
        const uint64_t x = (uint64_t)t * 256 + d;
        const uint32_t v = ly.hist[x];
        ly.hist[x] = run;
        run += v;
    }
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// A digit's counts over the tiles before `tile` and over all tiles, from its
// 16-bit row of nq 16-byte words (8 tiles each, padding zero).  All N loads
// are issued before any is used (indices past the row reread its last word
// and are not counted), so the row costs one memory round trip.
template <uint32_t N>
__device__ inline void row_sums(const uint4 *col, uint32_t nq, uint32_t tile, uint32_t &before, uint32_t &total)
{
    const u16x2 ones = {1, 1};
    uint4 v[N];
#pragma unroll
    for (uint32_t q = 0; q < N; q++) v[q] = col[min(q, nq - 1)];
#pragma unroll
    for (uint32_t q = 0; q < N; q++) {
        const uint32_t w[4] = {v[q].x, v[q].y, v[q].z, v[q].w};
        uint32_t sum = 0;
#pragma unroll
        for (int i = 0; i < 4; i++) sum = __builtin_amdgcn_udot2(__builtin_bit_cast(u16x2, w[i]), ones, sum, false);
        const uint32_t t = 8 * q;
        total += q < nq ? sum : 0u;
        uint32_t part = 0;  // counts of the tiles before `tile` among these 8 (a uniform branch)
        if (t + 8 <= tile) {
            part = sum;
        } else if (t < tile) {
#pragma unroll
            for (uint32_t i = 0; i < 8; i++) part += t + i < tile ? (w[i >> 1] >> (16 * (i & 1))) & 0xFFFFu : 0u;
        }
        before += q < nq ? part : 0u;
    }
}

// Stable scatter of one tile.  Thread tid owns digit tid: it reads the
// digit's 16-bit histogram row (16-byte loads, issued with the tile's keys) and
// sums the counts of the tiles before this one and of all tiles; a
// wave-level scan of the totals over digits gives the digit's base, so the
// tile's first destination for the digit is base + earlier tiles' count.
// A pass whose digit is the same for every element (some total equals n) is
// a no-op; every block takes that decision alike.  Element e = 256 u + tid
// of the tile is step u of its thread.  Every wave ranks its elements among
// equal digits of the same step with 8 ballots (one per digit bit) and
// records, per step and digit, how many it holds; after one barrier a
// thread per digit turns the counts, in (step, wave) order, into
// destination offsets; after a second barrier every element is written to
// offset + rank.  Block 0 records the result buffer for the next pass and
// in sort_cur (read only after the sort).  Without OWN_PREFIX, k_scan has
// turned the tile-major histogram into each (tile, digit)'s first
// destination and decided the skip.
template <bool OWN_PREFIX>
__global__ void __launch_bounds__(SORT_THREADS) k_scatter(Layout ly, uint64_t n, int shift, uint32_t tiles, int tgate,
                                                          uint32_t pass)
{
    constexpr uint32_t NW = SORT_THREADS / 64;
    __shared__ uint32_t off[SORT_PER][NW][256];  // counts, then offsets, per (step, wave, digit)
    __shared__ uint32_t wsum[NW];
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, tile = blockIdx.x;
    const uint32_t src = ly.ctl->sort_buf[pass];
    const bool lead = tile == 0 && tid == 0;
    if (!pass_active(ly, tgate) || (!OWN_PREFIX && ly.ctl->sort_skip)) {
        if (lead) ly.ctl->sort_buf[pass + 1] = ly.ctl->sort_cur = src;
        return;
    }
    const uint64_t *kin = ly.skey[src];
    const uint32_t *vin = ly.sval[src];
    uint64_t *kout = ly.skey[src ^ 1u];
    uint32_t *vout = ly.sval[src ^ 1u];
    const uint64_t base = (uint64_t)tile * SORT_TILE;
    uint64_t kk[SORT_PER];
    uint32_t vv[SORT_PER];
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++) {
        const uint64_t i = min(base + u * SORT_THREADS + tid, n - 1);
        kk[u] = kin[i];
        vv[u] = vin[i];
    }
    // digit tid over the tiles: before this one, and all
    const uint32_t hs = hist_stride(tiles);
    uint32_t before = 0, total = 0;
    if (OWN_PREFIX) {
        const uint4 *col =
            reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(ly.hist) + (uint64_t)tid * hs);
        static_assert(OWN_PREFIX_TILES <= 256, "a row is at most 32 loads");
        if (hs <= 64)
            row_sums<8>(col, hs / 8, tile, before, total);
        else
            row_sums<32>(col, hs / 8, tile, before, total);
    } else {
        before = ly.hist[(uint64_t)tile * 256 + tid];
    }
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++)
        for (uint32_t w = 0; w < NW; w++) off[u][w][tid] = 0;
    // inclusive scan of the totals over the wave's 64 digits
    uint32_t inc = total;
    for (uint32_t o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o);
        if (lane >= o) inc += y;
    }
    if (lane == 63) wsum[wave] = inc;
    if (__syncthreads_or(OWN_PREFIX && total == (uint32_t)n)) {
        if (lead) ly.ctl->sort_buf[pass + 1] = ly.ctl->sort_cur = src;
        return;
    }
    uint32_t run0 = inc - total + before;  // without OWN_PREFIX: total = inc = 0
    for (uint32_t w = 0; w < wave; w++) run0 += wsum[w];
    const uint64_t lt = (1ull << lane) - 1ull;
    uint8_t rk[SORT_PER];
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++) {
        const bool valid = base + u * SORT_THREADS + tid < n;
        const uint32_t dg = (uint32_t)(kk[u] >> shift) & 255u;
        uint64_t same = __ballot(valid);
        for (int b = 0; b < 8; b++) {
            const bool bit = (dg >> b) & 1u;
            const uint64_t bb = __ballot(bit);
            same &= bit ? bb : ~bb;
        }
        const uint32_t r = __popcll(same & lt);
        rk[u] = (uint8_t)r;
        if (valid && r == 0) off[u][wave][dg] = __popcll(same);
    }
    __syncthreads();
    // thread tid = digit: running offsets over (step, wave) in element order
    uint32_t run = run0;
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++)
        for (uint32_t w = 0; w < NW; w++) {
            const uint32_t c = off[u][w][tid];
            off[u][w][tid] = run;
            run += c;
        }
    __syncthreads();
#pragma unroll
    for (uint32_t u = 0; u < SORT_PER; u++) {
        if (base + u * SORT_THREADS + tid >= n) continue;
        const uint32_t dg = (uint32_t)(kk[u] >> shift) & 255u;
        const uint32_t dst = off[u][wave][dg] + rk[u];
        kout[dst] = kk[u];
        vout[dst] = vv[u];
    }
    if (lead) ly.ctl->sort_buf[pass + 1] = ly.ctl->sort_cur = src ^ 1u;
}

__global__ void k_sort_reset(Layout ly) { ly.ctl->sort_cur = 0; }

// The whole sort of at most one tile (SORT_TILE elements) in one workgroup:
// keys and values stay in LDS for all passes (ping-pong), each pass counts
// digits, scans them and scatters stably (ranks among equal digits by
// ballots per 256-element step, as in k_scatter); a pass whose digit is the
// same for every element is skipped.  The result is written back to the
// current buffer (buffer 0 after a reset), so the buffer index does not
// change.  Only the ceil(n / 256) steps that hold elements are worked.
// time_gate: byte b of the range is a start-time byte and runs only if the
// collective time reaches it (pass_active with tgate = 8 (b - byte_lo)).
__global__ void __launch_bounds__(SORT_THREADS) k_sort_small(Layout ly, uint32_t n, int byte_lo, int byte_hi,
                                                             bool reset_cur, bool time_gate)
{
    constexpr uint32_t NW = SORT_THREADS / 64;
    __shared__ uint64_t key[2][SORT_TILE];
    __shared__ uint32_t val[2][SORT_TILE];
    __shared__ uint32_t cnt[256];
    __shared__ uint16_t wc[SORT_PER][NW][256];  // counts, then offsets (below SORT_TILE)
    static_assert(SORT_TILE <= 65536, "offsets are 16-bit");
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t cur = reset_cur ? 0u : ly.ctl->sort_cur;
    if (reset_cur && tid == 0) ly.ctl->sort_cur = 0;
    const uint32_t steps = (n + SORT_THREADS - 1) / SORT_THREADS;
    for (uint32_t e = tid; e < n; e += SORT_THREADS) {
        key[0][e] = ly.skey[cur][e];
        val[0][e] = ly.sval[cur][e];
    }
    uint32_t b = 0;  // buffer holding the current order
    const uint64_t lt = (1ull << lane) - 1ull;
    for (int by = byte_lo; by < byte_hi; by++) {
        if (!pass_active(ly, time_gate ? 8 * (by - byte_lo) : -1)) break;
        const int shift = 8 * by;
        cnt[tid] = 0;
        for (uint32_t u = 0; u < steps; u++)
            for (uint32_t w = 0; w < NW; w++) wc[u][w][tid] = 0;
        __syncthreads();
        // ranks among equal digits inside each (step, wave), and their counts
        uint8_t rk[SORT_PER];
#pragma unroll
        for (uint32_t u = 0; u < SORT_PER; u++) {
            if (u >= steps) break;
            const uint32_t e = u * SORT_THREADS + tid;
            const bool valid = e < n;
            const uint32_t dg = valid ? (uint32_t)(key[b][e] >> shift) & 255u : 0u;
            uint64_t same = __ballot(valid);
            for (int bit = 0; bit < 8; bit++) {
                const bool x = (dg >> bit) & 1u;
                const uint64_t bb = __ballot(x);
                same &= x ? bb : ~bb;
            }
            const uint32_t r = __popcll(same & lt);
            rk[u] = (uint8_t)r;
            if (valid && r == 0) {
                wc[u][wave][dg] = (uint16_t)__popcll(same);
                atomicAdd(&cnt[dg], (uint32_t)__popcll(same));
            }
        }
        // one digit for every element: the pass is a no-op
        if (__syncthreads_or(cnt[tid] == n)) continue;
        // exclusive scan of the digit counts (Hillis-Steele), then offsets
        // per (step, wave) in element order for digit tid
        uint32_t v = cnt[tid];
        __syncthreads();
        for (uint32_t off = 1; off < 256; off <<= 1) {
            const uint32_t x = tid >= off ? cnt[tid - off] : 0u;
            __syncthreads();
            cnt[tid] += x;
            __syncthreads();
        }
        uint32_t run = cnt[tid] - v;
        for (uint32_t u = 0; u < steps; u++)
            for (uint32_t w = 0; w < NW; w++) {
                const uint32_t c = wc[u][w][tid];
                wc[u][w][tid] = (uint16_t)run;
                run += c;
            }
        __syncthreads();
#pragma unroll
        for (uint32_t u = 0; u < SORT_PER; u++) {
            const uint32_t e = u * SORT_THREADS + tid;
            if (e >= n) break;
            const uint32_t dg = (uint32_t)(key[b][e] >> shift) & 255u;
            const uint32_t dst = wc[u][wave][dg] + rk[u];
            key[b ^ 1u][dst] = key[b][e];
            val[b ^ 1u][dst] = val[b][e];
        }
        b ^= 1u;
        __syncthreads();
    }
    for (uint32_t e = tid; e < n; e += SORT_THREADS) {
        ly.skey[cur][e] = key[b][e];
        ly.sval[cur][e] = val[b][e];
    }
}

// Send log -> schedule.  Log key = t_start << 32 | link, value = rank.
// `add_cstar` shifts start times by the copy schedule's collective time
// (the All-Gather half of an All-Reduce).
__global__ void k_out_copy(Layout ly, uint64_t n, uint64_t out_off, uint32_t add_cstar, uint32_t flags)
{
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n || !log_complete(ly)) return;
    const uint32_t cur = ly.ctl->sort_cur;
    const uint64_t k = ly.skey[cur][i];
    const uint32_t r = ly.sval[cur][i];
    uint4 rec;
    rec.x = (uint32_t)k;
    rec.y = ly.order[r];
    rec.z = (uint32_t)(k >> 32) + (add_cstar ? ly.ctl->cstar : 0u);
    rec.w = flags;
    reinterpret_cast<uint4 *>(ly.out)[out_off + i] = rec;
}

// Forward log -> time-reversed keys (in place in the current buffer):
// (l, c, t) -> (reverse(l), c, C* - t - T[l]).
__global__ void k_reverse_keys(Layout ly, uint64_t n)
{
    uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n || !log_complete(ly)) return;
    const uint32_t cur = ly.ctl->sort_cur;
    const uint64_t k = ly.skey[cur][i];
    const uint32_t l = (uint32_t)k, t = (uint32_t)(k >> 32);
    const uint32_t tr = ly.ctl->cstar - t - ly.ltime[l];
    ly.skey[cur][i] = ((uint64_t)tr << 32) | ly.lrev[l];
}

}  // namespace

hipError_t radix_sort_pairs(const Layout &ly, uint64_t n, int byte_lo, int byte_hi, uint32_t max_tiles,
                            bool reset_cur, hipStream_t st, bool time_gate)
{
    if (n && n <= SORT_TILE) {
        k_sort_small<<<1, SORT_THREADS, 0, st>>>(ly, (uint32_t)n, byte_lo, byte_hi, reset_cur, time_gate);
        return hipGetLastError();
    }
    if (n == 0 || byte_hi <= byte_lo) {
        if (reset_cur) k_sort_reset<<<1, 1, 0, st>>>(ly);
        return hipGetLastError();
    }
    const uint32_t tiles = (uint32_t)((n + SORT_TILE - 1) / SORT_TILE);
    if (tiles > max_tiles || byte_hi - byte_lo > 8) return hipErrorInvalidValue;
    for (int b = byte_lo; b < byte_hi; b++) {
        const int tgate = time_gate ? 8 * (b - byte_lo) : -1;
        const uint32_t pass = (uint32_t)(b - byte_lo);
        if (tiles <= OWN_PREFIX_TILES) {
            k_hist<true><<<tiles, SORT_THREADS, 0, st>>>(ly, n, 8 * b, tiles, tgate, pass, reset_cur);
            k_scatter<true><<<tiles, SORT_THREADS, 0, st>>>(ly, n, 8 * b, tiles, tgate, pass);
        } else {
            k_hist<false><<<tiles, SORT_THREADS, 0, st>>>(ly, n, 8 * b, tiles, tgate, pass, reset_cur);
            k_scan<<<1, 256 * SCAN_SPLIT, 0, st>>>(ly, n, tiles, tgate);
            k_scatter<false><<<tiles, SORT_THREADS, 0, st>>>(ly, n, 8 * b, tiles, tgate, pass);
        }
    }
    return hipGetLastError();
}

static int bytes_for(uint64_t maxval)
{
    int b = 0;
    while (maxval) {
        b++;
        maxval >>= 8;
    }
    return b ? b : 1;
}

// Output stage: the send log (n entries, key t_start << 32 | link, value
// rank) is in sort buffer 0.  Writes the canonical schedule to ly.out.
// n is the number of deliveries the setup counted; the kernels may be
// queued before the matching kernel has run, so the collective time is
// read on the device and nothing is written unless the log is complete.
hipError_t launch_output(const Layout &ly, const Sizes &sz, int op, uint64_t n, hipStream_t st)
{
    // only the significant bytes of the link id (low word) and of the start
    // time (high word, start times are below the collective time) are sorted
    const int link_bytes = bytes_for(sz.L ? sz.L - 1 : 0);
    const int time_bytes = 4;  // passes past the collective time's bytes are gated off
    const int threads = 256;
    const uint64_t blocks = (n + threads - 1) / threads;
    hipError_t e;
    if (op == 0 || op == 2) {
        // forward schedule sorted by (t_start, link)
        e = radix_sort_pairs(ly, n, 0, link_bytes, sz.max_tiles, true, st);
        if (e != hipSuccess) return e;
        e = radix_sort_pairs(ly, n, 4, 4 + time_bytes, sz.max_tiles, false, st, true);
        if (e != hipSuccess) return e;
        if (n) {
            if (op == 0)
                k_out_copy<<<blocks, threads, 0, st>>>(ly, n, 0, 0, 0);
            else
                k_out_copy<<<blocks, threads, 0, st>>>(ly, n, n, 1, 0);
        }
    } else {
        k_sort_reset<<<1, 1, 0, st>>>(ly);
    }
    if (op == 1 || op == 2) {
        if (n) k_reverse_keys<<<blocks, threads, 0, st>>>(ly, n);
        e = radix_sort_pairs(ly, n, 0, link_bytes, sz.max_tiles, false, st);
        if (e != hipSuccess) return e;
        e = radix_sort_pairs(ly, n, 4, 4 + time_bytes, sz.max_tiles, false, st, true);
        if (e != hipSuccess) return e;
        if (n) k_out_copy<<<blocks, threads, 0, st>>>(ly, n, 0, 0, 1);
    }
    return hipGetLastError();
}

}  // namespace pccl
