// Setup of one synthesis on the device: conditions from the pre/postcondition
// bitmaps, shortest-path trees from every chunk source, condition distances,
// the priority order, relay devices and the initial holds/needs bitmaps over
// priority-ordered columns.
#include "pccl_internal.h"

namespace pccl {
namespace {

constexpr uint32_t FLAG_POST = 0x80000000u;  // holder_cnt: chunk has a postcondition bit
constexpr uint32_t CNT_MASK = 0x7FFFFFFFu;

// detail codes carried in error_arg[2] for PCCL_EINVAL
enum : uint32_t { BAD_TAIL = 1, BAD_MEMBER = 2, BAD_GROUP = 3, TWO_HOLDERS = 4, NO_HOLDER = 5 };

__global__ void k_fill32(uint32_t *p, uint64_t n, uint32_t v)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_fill64(uint64_t *p, uint64_t n, uint64_t v)
{
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

__global__ void k_ctl_reset(Control *ctl, unsigned long long max_sends)
{
    Control c = {};
    c.max_sends = max_sends;
    *ctl = c;
}

// Mask of valid bits in word k of a chunk row.
__device__ inline uint64_t tail_mask(uint64_t k, const Sizes &sz)
{
    if (k + 1 < sz.W || (sz.C & 63u) == 0) return NONE64;
    return (1ull << (sz.C & 63u)) - 1ull;
}

// Conditions (Sec. 4.1): for every set bit of the NPU-centric bitmaps,
// count precondition holders per chunk, mark chunks that are needed
// somewhere, and check that pre/post bits sit on members of the chunk's
// process group.  Grid: x over words, y over NPU rows.  The per-bit updates
// are atomics whose results are not used (a second holder is found by
// k_chunk_check), so a word's updates are in flight together; with a single
// process group the membership of the row is checked once per word.
__global__ void k_conditions(Layout ly, Sizes sz, const uint64_t *pre, const uint64_t *post,
                             const uint16_t *cg)
{
    const uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t v = blockIdx.y;
    if (k >= sz.W) return;
    const uint64_t p = pre[(uint64_t)v * sz.W + k], q = post[(uint64_t)v * sz.W + k];
    if (!(p | q)) return;
    const uint64_t tm = tail_mask(k, sz);
    if ((p | q) & ~tm) record_error(ly.ctl, ST_EINVAL, sz.C, v, BAD_TAIL);
    const uint64_t bits = (p | q) & tm;
    if (!cg) {
        if (bits && !((ly.group_masks[v >> 6] >> (v & 63)) & 1ull))
            record_error(ly.ctl, ST_EINVAL, (uint32_t)(k * 64 + __builtin_ctzll(bits)), v, BAD_MEMBER);
    } else {
        for (uint64_t x = bits; x; x &= x - 1) {
            const uint32_t c = (uint32_t)(k * 64 + __builtin_ctzll(x));
            const uint32_t g = cg[c];
            if (g >= sz.G) {
                record_error(ly.ctl, ST_EINVAL, c, v, BAD_GROUP);
                continue;
            }
            if (!((ly.group_masks[(uint64_t)g * sz.WN + (v >> 6)] >> (v & 63)) & 1ull))
                record_error(ly.ctl, ST_EINVAL, c, v, BAD_MEMBER);
        }
    }
    for (uint64_t x = p & tm; x; x &= x - 1) {
        const uint32_t c = (uint32_t)(k * 64 + __builtin_ctzll(x));
        atomicAdd(&ly.holder_cnt[c], 1u);
        ly.chunk_src[c] = v;  // the one holder (several are an error, reported below)
    }
    for (uint64_t x = q & tm; x; x &= x - 1) {
        const uint32_t c = (uint32_t)(k * 64 + __builtin_ctzll(x));
        atomicOr(&ly.holder_cnt[c], FLAG_POST);
    }
}

__global__ void k_chunk_check(Layout ly, Sizes sz)
{
    const uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= sz.C) return;
    const uint32_t h = ly.holder_cnt[c];
    if ((h & FLAG_POST) && !(h & CNT_MASK)) record_error(ly.ctl, ST_EINVAL, (uint32_t)c, 0, NO_HOLDER);
    if ((h & CNT_MASK) > 1u) record_error(ly.ctl, ST_EINVAL, (uint32_t)c, ly.chunk_src[c], TWO_HOLDERS);
    if ((h & CNT_MASK) == 1u) ly.src_index[ly.chunk_src[c]] = 1u;
}

// Distinct sources -> dense rows of the shortest-path tables (one workgroup).
__global__ void __launch_bounds__(1024) k_compact_sources(Layout ly, Sizes sz)
{
    __shared__ uint32_t part[1024];
    const uint32_t tid = threadIdx.x;
    const uint32_t per = (sz.N + 1023) / 1024;
    const uint32_t lo = tid * per, hi = min(lo + per, sz.N);
    uint32_t s = 0;
    for (uint32_t v = lo; v < hi; v++) s += ly.src_index[v];
    part[tid] = s;
    __syncthreads();
    for (uint32_t off = 1; off < 1024; off <<= 1) {
        uint32_t x = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += x;
        __syncthreads();
    }
    uint32_t run = tid ? part[tid - 1] : 0;
    for (uint32_t v = lo; v < hi; v++) {
        if (ly.src_index[v]) {
            ly.src_list[run] = v;
            ly.src_index[v] = run++;
        } else {
            ly.src_index[v] = NONE32;
        }
    }
    if (tid == 1023) ly.ctl->n_sources = part[1023];
}

constexpr uint32_t SP_BATCH = 8;  // links whose loads one thread issues together

// Shortest paths from one source per workgroup (Alg. 3 ShortestPath over
// the alpha-beta link times): Bellman-Ford relaxation with the distances in
// LDS, then the parent of each device = the smallest-id in-neighbour on a
// shortest path (the tree the pruned BFS of Sec. 4.3 keeps).
__global__ void __launch_bounds__(512) k_shortest_paths(Layout ly, Sizes sz)
{
    extern __shared__ unsigned long long dist[];
    __shared__ uint32_t changed;
    const uint32_t b = blockIdx.x, tid = threadIdx.x;
    if (b >= ly.ctl->n_sources || ly.ctl->error) return;
    const uint32_t s = ly.src_list[b];
    for (uint32_t v = tid; v < sz.D; v += blockDim.x) dist[v] = v == s ? 0ull : NONE64;
    __syncthreads();
    for (uint32_t it = 0; it < sz.D; it++) {
        if (tid == 0) changed = 0;
        __syncthreads();
        // eight links per thread loaded together (indices past L reread the
        // last link and are skipped)
        for (uint32_t e0 = tid; e0 < sz.L; e0 += SP_BATCH * blockDim.x) {
            uint32_t ls[SP_BATCH], ld[SP_BATCH], lt[SP_BATCH];
#pragma unroll
            for (uint32_t k = 0; k < SP_BATCH; k++) {
                const uint32_t e = min(e0 + k * blockDim.x, sz.L - 1u);
                ls[k] = ly.lsrc[e];
                ld[k] = ly.ldst[e];
                lt[k] = ly.ltime[e];
            }
#pragma unroll
            for (uint32_t k = 0; k < SP_BATCH; k++) {
                if (e0 + k * blockDim.x >= sz.L) continue;
                const unsigned long long du = dist[ls[k]];
                if (du == NONE64) continue;
                const unsigned long long nd = du + lt[k];
                if (nd < dist[ld[k]]) {
                    atomicMin(&dist[ld[k]], nd);
                    changed = 1;
                }
            }
        }
        __syncthreads();
        const uint32_t again = changed;
        __syncthreads();
        if (!again) break;
    }
    for (uint32_t v = tid; v < sz.D; v += blockDim.x) {
        const unsigned long long dv = dist[v];
        ly.sp_dist[(uint64_t)b * sz.D + v] = dv;
        uint32_t par = NONE32;
        if (v != s && dv != NONE64) {
            const uint32_t i0 = ly.in_off[v], i1 = ly.in_off[v + 1];
            for (uint32_t i = i0; i < i1; i += SP_BATCH) {
                uint32_t su[SP_BATCH], st[SP_BATCH];
#pragma unroll
                for (uint32_t k = 0; k < SP_BATCH; k++) {
                    const uint32_t x = min(i + k, i1 - 1u);
                    su[k] = ly.slot_src[x];
                    st[k] = ly.slot_time[x];
                }
#pragma unroll
                for (uint32_t k = 0; k < SP_BATCH; k++) {
                    if (i + k >= i1) continue;
                    const unsigned long long du = dist[su[k]];
                    if (du != NONE64 && du + st[k] == dv && su[k] < par) par = su[k];
                }
            }
        }
        ly.sp_parent[(uint64_t)b * sz.D + v] = par;
    }
}

// Condition distance = max over destinations of the shortest-path distance
// (Alg. 3); destinations = postcondition and not precondition.
__global__ void k_chunk_dist(Layout ly, Sizes sz, const uint64_t *pre, const uint64_t *post)
{
    if (ly.ctl->error) return;
    const uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t v = blockIdx.y;
    if (k >= sz.W) return;
    const uint64_t x0 = post[(uint64_t)v * sz.W + k] & ~pre[(uint64_t)v * sz.W + k] & tail_mask(k, sz);
    for (uint64_t x = x0; x; x &= x - 1) {
        const uint32_t c = (uint32_t)(k * 64 + __builtin_ctzll(x));
        const uint32_t row = ly.src_index[ly.chunk_src[c]];
        const unsigned long long dv = ly.sp_dist[(uint64_t)row * sz.D + v];
        if (dv == NONE64)
            record_error(ly.ctl, ST_EUNREACHABLE, c, v, ly.chunk_src[c]);
        else if (dv >= 0xFFFFFFFFull)
            record_error(ly.ctl, ST_ERANGE, c, v, 1);
        else
            atomicMax(&ly.chunk_dist[c], dv);
    }
}

// Switch model: for every limited-switch row and chunk rank, how many of the
// switch's out-links lead to a device that needs the chunk once the needs
// rows are set up (the matching kernel keeps the count as those devices
// receive it, and reads it when the switch takes the chunk into a buffer
// place).  One thread per (row, chunk): the 64 threads of a wave read the
// same needs word of each out-neighbour.
__global__ void k_adm_counts(Layout ly, Sizes sz)
{
    const uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t row = blockIdx.y;
    if (c >= sz.C) return;
    const uint32_t o0 = ly.sw.b_abs[2 * row], no = ly.sw.b_abs[2 * row + 1];
    uint32_t n = 0;
    for (uint32_t q = 0; q < no; q++) {
        const uint32_t o = ly.sw.b_out[o0 + q] & 0xFFFFu;
        n += (uint32_t)((ly.needs[(uint64_t)o * sz.Wp + (c >> 6)] >> (c & 63u)) & 1ull);
    }
    ly.sw.acnt[(uint64_t)row * sz.C + c] = n;
}

// Priority order (distance descending, then the SplitMix64 key ascending,
// then chunk id): one stable sort of the bitwise-not of the distance (high
// word) and the key's high word (low word), from chunk id order, then runs
// of equal sort keys ordered by the key's low word (k_key_ties).
__global__ void k_keys_hash(Layout ly, Sizes sz, uint64_t seed)
{
    const uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= sz.C) return;
    const uint32_t nd = ~(uint32_t)ly.chunk_dist[c];
    ly.skey[0][c] = ((uint64_t)nd << 32) | (splitmix64_key(seed, c) >> 32);
    ly.sval[0][c] = (uint32_t)c;
}

// After the sort: the first thread of a run of equal sort keys (equal
// distance and key high word; with random keys a run is rare and short)
// orders the run by (key low word, chunk id), in place.
__global__ void k_key_ties(Layout ly, Sizes sz, uint64_t seed)
{
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= sz.C) return;
    const uint32_t cur = ly.ctl->sort_cur;
    const uint64_t *k = ly.skey[cur];
    uint32_t *v = ly.sval[cur];
    const uint64_t ki = k[i];
    if ((i > 0 && k[i - 1] == ki) || i + 1 >= sz.C || k[i + 1] != ki) return;
    uint64_t j = i + 2;
    while (j < sz.C && k[j] == ki) j++;
    // insertion sort; the stable sort left the run in chunk id order
    for (uint64_t a = i + 1; a < j; a++) {
        const uint32_t c = v[a], lo = (uint32_t)splitmix64_key(seed, c);
        uint64_t b = a;
        while (b > i) {
            const uint32_t p = v[b - 1], plo = (uint32_t)splitmix64_key(seed, p);
            if (plo < lo || (plo == lo && p < c)) break;
            v[b] = p;
            b--;
        }
        v[b] = c;
    }
}

__global__ void k_rank(Layout ly, Sizes sz)
{
    const uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= sz.C) return;
    const uint32_t c = ly.sval[ly.ctl->sort_cur][r];
    ly.order[r] = c;
    ly.rank[c] = (uint32_t)r;
}

__global__ void k_holds(Layout ly, Sizes sz)
{
    if (ly.ctl->error) return;
    const uint64_t c = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= sz.C) return;
    if ((ly.holder_cnt[c] & CNT_MASK) != 1u) return;
    const uint32_t r = ly.rank[c];
    atomicOr((unsigned long long *)&ly.holds[(uint64_t)ly.chunk_src[c] * sz.Wp + (r >> 6)], 1ull << (r & 63));
}

// needs = destinations plus the relays on their tree paths (the paths the
// pruned BFS keeps, Sec. 4.3): walk parents from each destination up to the
// source.  A walk that meets a bit already set stops there: whoever set it
// is a destination or a walk that continues upward.  Two walks may both
// pass a device before either bit is visible; both then set it (harmless).
__global__ void k_needs(Layout ly, Sizes sz, const uint64_t *pre, const uint64_t *post)
{
    if (ly.ctl->error) return;
    const uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint32_t v = blockIdx.y;
    if (k >= sz.W) return;
    const uint64_t x0 = post[(uint64_t)v * sz.W + k] & ~pre[(uint64_t)v * sz.W + k] & tail_mask(k, sz);
    for (uint64_t x = x0; x; x &= x - 1) {
        const uint32_t c = (uint32_t)(k * 64 + __builtin_ctzll(x));
        const uint32_t s = ly.chunk_src[c], row = ly.src_index[s], r = ly.rank[c];
        const uint64_t bit = 1ull << (r & 63);
        const uint32_t *par = ly.sp_parent + (uint64_t)row * sz.D;
        uint32_t u = v;
        for (uint32_t hop = 0; hop < sz.D && u != s && u < sz.D; hop++) {
            unsigned long long *w = (unsigned long long *)&ly.needs[(uint64_t)u * sz.Wp + (r >> 6)];
            const uint32_t next = par[u];
            // a relay bit another walk already set: that walk covers the rest
            if ((atomicOr(w, bit) & bit) && hop > 0) break;
            u = next;
        }
    }
}

// Candidates of every link at the start (one wave per destination-major
// slot): popcount(holds[src] & needs[dst]) over the rows.  The matching
// kernel keeps this count as an upper bound (arrivals add, the link's own
// commits subtract, a pick round that finds nothing resets it to 0), so a
// freed link whose bound is 0 has no candidate and needs no scan.
__global__ void __launch_bounds__(256) k_link_counts(Layout ly, Sizes sz)
{
    if (ly.ctl->error) return;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t sl = (uint64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (sl >= sz.L) return;
    const uint64_t Ws = (sz.W + 1) & ~1ull;
    const uint64_t *h = ly.holds + (uint64_t)ly.slot_src[sl] * sz.Wp;
    const uint64_t *n = ly.needs + (uint64_t)ly.ldst[ly.slot_link[sl]] * sz.Wp;
    uint32_t c = 0;
    for (uint64_t w = 2 * lane; w < Ws; w += 128) {
        const uint4 a = *reinterpret_cast<const uint4 *>(h + w), b = *reinterpret_cast<const uint4 *>(n + w);
        c += __popc(a.x & b.x) + __popc(a.y & b.y) + __popc(a.z & b.z) + __popc(a.w & b.w);
    }
    for (int off = 32; off; off >>= 1) c += (uint32_t)__shfl_xor((int)c, off);
    if (lane == 0) ly.lcnt[sl] = c;
}

// Each destination gets a contiguous segment of the send log, as long as
// the number of deliveries it needs (every delivery is one transfer into it).
__global__ void __launch_bounds__(256) k_needs_count(Layout ly, Sizes sz)
{
    __shared__ unsigned long long part[4];
    const uint32_t d = blockIdx.x, tid = threadIdx.x;
    unsigned long long c = 0;
    if (!ly.ctl->error) {
        const uint64_t *row = ly.needs + (uint64_t)d * sz.Wp;
        for (uint64_t w = tid; w < sz.Wp; w += 256) c += (unsigned long long)__popcll(row[w]);
    }
    for (int off = 32; off; off >>= 1) c += __shfl_xor(c, off);
    if ((tid & 63) == 0) part[tid >> 6] = c;
    __syncthreads();
    if (tid == 0) ly.dest_log[d] = part[0] + part[1] + part[2] + part[3];
}

__global__ void __launch_bounds__(1024) k_log_offsets(Layout ly, Sizes sz)
{
    __shared__ unsigned long long part[1024];
    const uint32_t tid = threadIdx.x;
    const uint32_t per = (sz.D + 1023) / 1024;
    const uint32_t lo = tid * per, hi = min(lo + per, sz.D);
    unsigned long long s = 0;
    for (uint32_t v = lo; v < hi; v++) s += ly.dest_log[v];
    part[tid] = s;
    __syncthreads();
    for (uint32_t off = 1; off < 1024; off <<= 1) {
        unsigned long long x = tid >= off ? part[tid - off] : 0;
        __syncthreads();
        part[tid] += x;
        __syncthreads();
    }
    unsigned long long run = tid ? part[tid - 1] : 0;
    for (uint32_t v = lo; v < hi; v++) {
        const unsigned long long c = ly.dest_log[v];
        ly.dest_log[v] = run;
        run += c;
    }
    if (tid == 1023) ly.ctl->needs_total = part[1023];
}

__global__ void k_init_match(Layout ly, Sizes sz)
{
    const uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < sz.L) {
        ly.busy[i] = 0;
        ly.infl[i] = NONE32;
        ly.cur[i] = 0;
        ly.lflags[i] = 0;
        ly.snap[i] = NONE64;
        ly.snap[sz.L + i] = NONE64;
        ly.snap[2ull * sz.L + i] = NONE64;
    }
    if (i < 2ull * MAX_MATCH_GRID) ly.xslot[i * XSLOT_WORDS] = 0;
    if (i == 0) {
        Control *ctl = ly.ctl;
        ctl->needs_remaining = ctl->needs_total;
        if (!ctl->error && ctl->needs_total > ctl->max_sends)
            record_error(ctl, ST_ENOMEM, (uint32_t)(ctl->needs_total >> 32), (uint32_t)ctl->needs_total, 0);
    }
}

inline uint32_t blocks_for(uint64_t n, uint32_t t) { return (uint32_t)((n + t - 1) / t); }

}  // namespace

hipError_t launch_setup(const Layout &ly, const Sizes &sz, const uint64_t *pre, const uint64_t *post,
                        const uint16_t *chunk_group, uint64_t seed, hipStream_t st)
{
    const uint32_t T = 256;
    k_ctl_reset<<<1, 1, 0, st>>>(ly.ctl, sz.max_sends);
    const uint64_t C = sz.C;
    if (C) {
        k_fill32<<<min(blocks_for(C, T), 4096u), T, 0, st>>>(ly.holder_cnt, C, 0);
        k_fill32<<<min(blocks_for(C, T), 4096u), T, 0, st>>>(ly.chunk_src, C, NONE32);
        k_fill64<<<min(blocks_for(C, T), 4096u), T, 0, st>>>(ly.chunk_dist, C, 0);
    }
    k_fill32<<<blocks_for(sz.N, T), T, 0, st>>>(ly.src_index, sz.N, 0);
    const uint64_t bm = (uint64_t)sz.D * sz.Wp;
    k_fill64<<<min(blocks_for(bm, T), 8192u), T, 0, st>>>(ly.holds, bm, 0);
    k_fill64<<<min(blocks_for(bm, T), 8192u), T, 0, st>>>(ly.needs, bm, 0);
    const dim3 gw(blocks_for(sz.W ? sz.W : 1, T), sz.N);
    if (sz.W) k_conditions<<<gw, T, 0, st>>>(ly, sz, pre, post, chunk_group);
    if (C) k_chunk_check<<<blocks_for(C, T), T, 0, st>>>(ly, sz);
    k_compact_sources<<<1, 1024, 0, st>>>(ly, sz);
    k_shortest_paths<<<sz.N, 512, sizeof(unsigned long long) * sz.D, st>>>(ly, sz);
    if (sz.W) k_chunk_dist<<<gw, T, 0, st>>>(ly, sz, pre, post);
    if (C) {
        k_keys_hash<<<blocks_for(C, T), T, 0, st>>>(ly, sz, seed);
        const hipError_t e = radix_sort_pairs(ly, C, 0, 8, sz.max_tiles, true, st);
        if (e != hipSuccess) return e;
        k_key_ties<<<blocks_for(C, T), T, 0, st>>>(ly, sz, seed);
        k_rank<<<blocks_for(C, T), T, 0, st>>>(ly, sz);
        k_holds<<<blocks_for(C, T), T, 0, st>>>(ly, sz);
    }
    if (sz.W) k_needs<<<gw, T, 0, st>>>(ly, sz, pre, post);
    if (sz.sw_nbt && C) k_adm_counts<<<dim3(blocks_for(C, T), sz.sw_nbt), T, 0, st>>>(ly, sz);
    if (sz.L) k_link_counts<<<blocks_for(sz.L, 4), 256, 0, st>>>(ly, sz);
    k_needs_count<<<sz.D, 256, 0, st>>>(ly, sz);
    k_log_offsets<<<1, 1024, 0, st>>>(ly, sz);
    k_init_match<<<blocks_for(std::max<uint64_t>(sz.L, 4ull * MAX_MATCH_GRID), T), T, 0, st>>>(ly, sz);
    return hipGetLastError();
}

}  // namespace pccl
