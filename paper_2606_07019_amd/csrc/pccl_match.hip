// The event-stepped chunk-to-link matching, as one persistent cooperative
// kernel.
//
// Semantics (what the schedule must equal): at every event time t, links
// whose transfer ends at t deliver and become free; then every free link
// s->d picks the highest-priority chunk held by s and still needed by d (the
// BFS step of Alg. 2, applied to all free links at once); picks that deliver
// the same chunk to the same device clash, the fastest link (then the lowest
// link id) wins and commits (the link is busy for its alpha-beta time,
// Sec. 4.4/4.6), losers pick again until nobody can pick; then time advances
// to the earliest transfer end (NextAvailableTime, Alg. 1).
//
// Execution (how the device reaches exactly that): two facts make the event
// loop parallel over destinations and coarse in time.
//  1. Within one event, picks into different destinations never interact:
//     holds do not change during an event and a commit only clears a bit of
//     its own destination's needs row.  So each destination device d is
//     owned by one workgroup, which keeps d's in-links, d's needs row and
//     the arrivals into d; clashes are resolved inside the workgroup.
//  2. A transfer started at time >= t0 ends no earlier than t0 + Tmin (the
//     smallest link time).  So every arrival inside [t0, t0 + Tmin) comes
//     from a transfer that started before t0 and is known when the window
//     starts.  All events of the window are processed without a global
//     synchronization; one grid barrier per window publishes the transfers
//     in flight (a per-link snapshot) and the next event time.
// Arrivals are folded into the owner's holds row one window late; readers
// add the last two snapshots explicitly, so every pick sees exactly the
// chunks that have arrived by its event time.
//
// Per-link scan state keeps the intersect work small: a free link whose
// candidate set was found empty stays empty until its source receives a
// chunk its destination needs (needs only shrink), so it is not rescanned;
// a busy link keeps a cursor below which it has no candidate (lowered when
// its source receives a needed chunk), so its next scan starts there.
#include "pccl_internal.h"

namespace pccl {
namespace {

constexpr uint32_t NT = MATCH_THREADS;
constexpr uint32_t NWAVES = NT / 64;
constexpr uint8_t M_IDLE = 0, M_FULL = 1, M_ARR = 2, M_ARR_WON = 3;
constexpr uint32_t SPIN_LIMIT = 1u << 22;

struct Shared {
    uint32_t link[MAX_IN_LINKS], src[MAX_IN_LINKS], tim[MAX_IN_LINKS];
    uint32_t busy[MAX_IN_LINKS], infl[MAX_IN_LINKS], cur[MAX_IN_LINKS], pick[MAX_IN_LINKS];
    uint32_t cum[MAX_IN_LINKS + 1];
    uint32_t full_list[MAX_IN_LINKS];
    uint8_t mode[MAX_IN_LINKS], idle[MAX_IN_LINKS], win[MAX_IN_LINKS];
    uint32_t arr_end[MAX_PAIRS], arr_c[MAX_PAIRS];
    uint16_t arr_j[MAX_PAIRS];
    uint32_t unf_c[MAX_PAIRS];
    uint16_t unf_j[MAX_PAIRS];
    uint32_t snd_link[MAX_IN_LINKS], snd_rank[MAX_IN_LINKS], snd_t[MAX_IN_LINKS];
    uint32_t n_arr, n_unf, n_full, n_send, send_base;
    uint32_t red[NWAVES];
    uint32_t barrier_ok;
};

__device__ inline bool need_bit(const uint64_t *nd, uint32_t c)
{
    return (nd[c >> 6] >> (c & 63)) & 1ull;
}

__device__ inline uint32_t block_min(uint32_t v, Shared &sh)
{
    for (int off = 32; off; off >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, off));
    if ((threadIdx.x & 63) == 0) sh.red[threadIdx.x >> 6] = v;
    __syncthreads();
    uint32_t r = sh.red[0];
    for (uint32_t w = 1; w < NWAVES; w++) r = min(r, sh.red[w]);
    __syncthreads();
    return r;
}

__device__ inline uint32_t block_or(uint32_t v, Shared &sh)
{
    const uint32_t any = __ballot(v != 0) != 0ull;
    if ((threadIdx.x & 63) == 0) sh.red[threadIdx.x >> 6] = any;
    __syncthreads();
    uint32_t r = 0;
    for (uint32_t w = 0; w < NWAVES; w++) r |= sh.red[w];
    __syncthreads();
    return r;
}

__device__ inline uint64_t shfl64(uint64_t v, int lane)
{
    const int lo = __shfl((int)(uint32_t)v, lane), hi = __shfl((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// Bitset intersect + select for one link, by a whole wave: the first set bit
// at position >= cur of holds[src] & needs[dst], in priority order.  Each
// lane loads 16 bytes of each row per sweep (two sweeps in flight, 2 KiB per
// row per wave), a ballot finds the first lane with a non-zero AND, and a
// count-trailing-zeros gives the chunk.
__device__ uint32_t wave_first_candidate(const uint64_t *__restrict__ h, const uint64_t *__restrict__ nd,
                                         uint32_t cur, uint64_t Wp, uint64_t &words)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t w0 = cur >> 6;
    if (w0 >= Wp) return NONE32;
    const uint64_t keep0 = ~0ull << (cur & 63);
    for (uint64_t wb = w0 & ~1ull; wb < Wp; wb += 256) {
        uint64_t a[2], b[2];
#pragma unroll
        for (int u = 0; u < 2; u++) {
            const uint64_t idx = wb + 128 * u + 2 * lane;
            uint64_t x = 0, y = 0;
            if (idx < Wp) {
                const uint4 hv = *reinterpret_cast<const uint4 *>(h + idx);
                const uint4 nv = *reinterpret_cast<const uint4 *>(nd + idx);
                x = (((uint64_t)hv.y << 32) | hv.x) & (((uint64_t)nv.y << 32) | nv.x);
                y = (((uint64_t)hv.w << 32) | hv.z) & (((uint64_t)nv.w << 32) | nv.z);
                if (idx < w0) x = 0;
                else if (idx == w0) x &= keep0;
                if (idx + 1 < w0) y = 0;
                else if (idx + 1 == w0) y &= keep0;
            }
            a[u] = x;
            b[u] = y;
        }
#pragma unroll
        for (int u = 0; u < 2; u++) {
            const uint64_t m = __ballot((a[u] | b[u]) != 0ull);
            if (m) {
                const int fl = __builtin_ffsll((long long)m) - 1;
                const uint64_t x = shfl64(a[u], fl), y = shfl64(b[u], fl);
                const uint64_t idx = wb + 128 * u + 2 * (uint64_t)fl;
                words += (x ? idx : idx + 1) + 1 - w0;
                return x ? (uint32_t)(idx * 64 + __builtin_ctzll(x))
                         : (uint32_t)((idx + 1) * 64 + __builtin_ctzll(y));
            }
        }
    }
    words += Wp - w0;
    return NONE32;
}

// Grid-wide barrier on a monotonic arrival counter.  Returns false when the
// wait timed out or another workgroup gave up (then the kernel ends).
__device__ bool grid_barrier(Control *ctl, Shared &sh)
{
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t nb = gridDim.x;
        uint32_t ok = 1;
        __threadfence();
        const uint32_t old = atomicAdd(&ctl->barrier, 1u);
        const uint32_t target = (old / nb + 1u) * nb;
        uint32_t spins = 0;
        while (true) {
            const uint32_t v = __hip_atomic_load(&ctl->barrier, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if ((int32_t)(v - target) >= 0) break;
            if (__hip_atomic_load(&ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                ok = 0;
                break;
            }
            if (++spins > SPIN_LIMIT) {
                atomicExch(&ctl->abort, 1u);
                ok = 0;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        __threadfence();
        sh.barrier_ok = ok;
    }
    __syncthreads();
    return sh.barrier_ok != 0;
}

__device__ inline void window_error(Control *ctl, uint32_t k, uint32_t code, uint32_t a, uint32_t b, uint32_t c)
{
    record_error(ctl, code, a, b, c);
    atomicOr(&ctl->win_err[k % 3], 1u);
}

struct Acc {
    uint32_t tmin;     // earliest end among transfers in flight (this thread's links)
    uint32_t cstar;    // latest transfer end committed by this thread
    uint32_t clashes;  // picks of this thread that lost a clash
    uint64_t words;    // words per row scanned by this thread's wave (lane 0)
};

// All events of window [t0, t1) for destination d.
__device__ void process_destination(const Layout &ly, const Sizes &sz, Shared &sh, uint32_t d, uint32_t k,
                                    uint32_t t0, uint64_t t1, Acc &acc, unsigned long long &rounds,
                                    unsigned long long &sent)
{
    const uint32_t tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const uint32_t base = ly.in_off[d], n = ly.in_off[d + 1] - base;
    if (n == 0) return;
    const uint64_t Wp = sz.Wp, L = sz.L;
    const uint32_t END = (uint32_t)(Wp * 64);
    uint64_t *nd = ly.needs + (uint64_t)d * Wp;
    uint64_t *hd = ly.holds + (uint64_t)d * Wp;
    const uint64_t *snap1 = ly.snap + (uint64_t)((k + 2) % 3) * L;  // in flight at the end of window k-1
    const uint64_t *snap2 = ly.snap + (uint64_t)((k + 1) % 3) * L;  // in flight at the end of window k-2
    uint64_t *snap0 = ly.snap + (uint64_t)(k % 3) * L;              // written for window k+1

    // load this destination's in-links; fold the arrivals of window k-1
    for (uint32_t i = tid; i < n; i += NT) {
        const uint32_t sl = base + i;
        sh.link[i] = ly.slot_link[sl];
        sh.src[i] = ly.slot_src[sl];
        sh.tim[i] = ly.slot_time[sl];
        sh.busy[i] = ly.busy[sl];
        sh.infl[i] = ly.infl[sl];
        sh.cur[i] = ly.cur[sl];
        sh.idle[i] = (uint8_t)(ly.lflags[sl] & 1u);
        sh.cum[i] = ly.slot_cum[sl];
        sh.mode[i] = M_IDLE;
        if (k >= 2) {
            const uint64_t e = snap2[sl];
            if (e != NONE64 && (uint32_t)e < t0) {
                const uint32_t r = (uint32_t)(e >> 32);
                atomicOr((unsigned long long *)&hd[r >> 6], 1ull << (r & 63));
            }
        }
    }
    if (tid == 0) {
        sh.n_arr = 0;
        sh.n_unf = 0;
        sh.n_send = 0;
        sh.cum[n] = ly.dest_pairs[d];
    }
    __syncthreads();

    // arrivals at the sources of d's in-links that d needs: this window's
    // (snapshot k-1, ends in [t0, t1)) and last window's (snapshot k-2,
    // ends before t0; possibly not folded into the source's row yet)
    const uint32_t pairs = sh.cum[n];
    if (k >= 1) {
        for (uint32_t p = tid; p < pairs; p += NT) {
            uint32_t lo = 0, hi = n;
            while (hi - lo > 1) {
                const uint32_t mid = (lo + hi) >> 1;
                if (sh.cum[mid] <= p) lo = mid;
                else hi = mid;
            }
            const uint32_t s = sh.src[lo];
            const uint32_t slot = ly.in_off[s] + (p - sh.cum[lo]);
            const uint64_t e1 = snap1[slot];
            if (e1 != NONE64 && (uint64_t)(uint32_t)e1 < t1) {
                const uint32_t c = (uint32_t)(e1 >> 32);
                if (need_bit(nd, c)) {
                    const uint32_t q = atomicAdd(&sh.n_arr, 1u);
                    sh.arr_end[q] = (uint32_t)e1;
                    sh.arr_c[q] = c;
                    sh.arr_j[q] = (uint16_t)lo;
                }
            }
            if (k >= 2) {
                const uint64_t e2 = snap2[slot];
                if (e2 != NONE64 && (uint32_t)e2 < t0) {
                    const uint32_t c = (uint32_t)(e2 >> 32);
                    if (need_bit(nd, c)) {
                        const uint32_t q = atomicAdd(&sh.n_unf, 1u);
                        sh.unf_c[q] = c;
                        sh.unf_j[q] = (uint16_t)lo;
                    }
                }
            }
        }
    }
    __syncthreads();
    const uint32_t n_arr = sh.n_arr, n_unf = sh.n_unf;

    // event times of this destination inside the window, in order
    int64_t t_prev = (int64_t)t0 - 1;
    while (true) {
        uint32_t m = NONE32;
        if (k == 0) {
            if (t_prev < 0 && tid == 0) m = 0;
        } else {
            for (uint32_t i = tid; i < n; i += NT)
                if (sh.infl[i] != NONE32 && (int64_t)sh.busy[i] > t_prev && (uint64_t)sh.busy[i] < t1)
                    m = min(m, sh.busy[i]);
            for (uint32_t q = tid; q < n_arr; q += NT)
                if ((int64_t)sh.arr_end[q] > t_prev) m = min(m, sh.arr_end[q]);
        }
        const uint32_t t = block_min(m, sh);
        if (t == NONE32) break;

        // links whose transfer ends now are free and need a full scan
        for (uint32_t i = tid; i < n; i += NT) {
            uint8_t md = M_IDLE;
            if (k == 0) {
                md = M_FULL;
            } else if (sh.infl[i] != NONE32 && sh.busy[i] == t) {
                md = M_FULL;
                sh.infl[i] = NONE32;
            }
            sh.mode[i] = md;
        }
        __syncthreads();
        // a needed chunk arriving at a link's source: busy or just-freed links
        // lower their cursor; an idle free link gets it as its candidate
        for (uint32_t q = tid; q < n_arr; q += NT) {
            if (sh.arr_end[q] != t) continue;
            const uint32_t j = sh.arr_j[q], c = sh.arr_c[q];
            if (!need_bit(nd, c)) continue;
            if (sh.mode[j] == M_FULL || sh.infl[j] != NONE32)
                atomicMin(&sh.cur[j], c);
            else if (sh.idle[j])
                sh.mode[j] = M_ARR;
        }
        __syncthreads();

        // pick rounds at time t
        while (true) {
            for (uint32_t i = tid; i < n; i += NT) sh.pick[i] = NONE32;
            if (tid == 0) sh.n_full = 0;
            __syncthreads();
            for (uint32_t i = tid; i < n; i += NT)
                if (sh.mode[i] == M_FULL) sh.full_list[atomicAdd(&sh.n_full, 1u)] = i;
            __syncthreads();
            const uint32_t nf = sh.n_full;
            for (uint32_t f = wave; f < nf; f += NWAVES) {
                const uint32_t j = sh.full_list[f];
                const uint32_t p =
                    wave_first_candidate(ly.holds + (uint64_t)sh.src[j] * Wp, nd, sh.cur[j], Wp, acc.words);
                if (lane == 0 && p != NONE32) atomicMin(&sh.pick[j], p);
            }
            for (uint32_t q = tid; q < n_arr; q += NT) {
                const uint32_t j = sh.arr_j[q], c = sh.arr_c[q], md = sh.mode[j];
                if (md == M_FULL) {
                    if (sh.arr_end[q] <= t && c >= sh.cur[j] && need_bit(nd, c)) atomicMin(&sh.pick[j], c);
                } else if (md == M_ARR) {
                    if (sh.arr_end[q] == t && need_bit(nd, c)) atomicMin(&sh.pick[j], c);
                }
            }
            for (uint32_t q = tid; q < n_unf; q += NT) {
                const uint32_t j = sh.unf_j[q], c = sh.unf_c[q];
                if (sh.mode[j] == M_FULL && c >= sh.cur[j] && need_bit(nd, c)) atomicMin(&sh.pick[j], c);
            }
            __syncthreads();
            uint32_t any = 0;
            for (uint32_t i = tid; i < n; i += NT) {
                if (sh.mode[i] == M_IDLE) continue;
                if (sh.pick[i] == NONE32) {
                    sh.mode[i] = M_IDLE;
                    sh.idle[i] = 1;
                    sh.cur[i] = END;
                } else {
                    any = 1;
                }
            }
            if (!block_or(any, sh)) break;
            // clash resolution among d's in-links: fastest link, then lowest id
            for (uint32_t i = tid; i < n; i += NT) {
                if (sh.mode[i] == M_IDLE) continue;
                const uint32_t p = sh.pick[i], ti = sh.tim[i], li = sh.link[i];
                uint8_t w = 1;
                for (uint32_t j = 0; j < n; j++) {
                    if (j == i || sh.mode[j] == M_IDLE || sh.pick[j] != p) continue;
                    if (sh.tim[j] < ti || (sh.tim[j] == ti && sh.link[j] < li)) w = 0;
                }
                sh.win[i] = w;
            }
            __syncthreads();
            for (uint32_t i = tid; i < n; i += NT) {
                if (sh.mode[i] == M_IDLE) continue;
                const uint32_t p = sh.pick[i];
                if (sh.win[i]) {
                    atomicAnd((unsigned long long *)&nd[p >> 6], ~(1ull << (p & 63)));
                    const uint64_t end = (uint64_t)t + sh.tim[i];
                    if (end > 0xFFFFFFFFull) window_error(ly.ctl, k, ST_ERANGE, p, d, 2);
                    const uint32_t e32 = end > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)end;
                    sh.infl[i] = p;
                    sh.busy[i] = e32;
                    sh.idle[i] = 0;
                    const uint32_t q = atomicAdd(&sh.n_send, 1u);
                    sh.snd_link[q] = sh.link[i];
                    sh.snd_rank[q] = p;
                    sh.snd_t[q] = t;
                    acc.cstar = max(acc.cstar, e32);
                    if (sh.mode[i] == M_FULL) {
                        sh.cur[i] = p + 1;
                        sh.mode[i] = M_IDLE;
                    } else {
                        sh.cur[i] = END;
                        sh.mode[i] = M_ARR_WON;
                    }
                } else {
                    acc.clashes++;
                    if (sh.mode[i] == M_FULL) sh.cur[i] = p + 1;
                }
            }
            __syncthreads();
            // a link that won an arrival keeps the other arrivals as its cursor
            for (uint32_t q = tid; q < n_arr; q += NT) {
                if (sh.arr_end[q] != t) continue;
                const uint32_t j = sh.arr_j[q], c = sh.arr_c[q];
                if (sh.mode[j] == M_ARR_WON && need_bit(nd, c)) atomicMin(&sh.cur[j], c);
            }
            __syncthreads();
            for (uint32_t i = tid; i < n; i += NT)
                if (sh.mode[i] == M_ARR_WON) sh.mode[i] = M_IDLE;
            if (tid == 0) rounds++;
            __syncthreads();
        }
        t_prev = t;
    }

    // write back link state and this window's snapshot
    for (uint32_t i = tid; i < n; i += NT) {
        const uint32_t sl = base + i;
        ly.busy[sl] = sh.busy[i];
        ly.infl[sl] = sh.infl[i];
        ly.cur[sl] = sh.cur[i];
        ly.lflags[sl] = sh.idle[i];
        if (sh.infl[i] != NONE32) {
            snap0[sl] = ((uint64_t)sh.infl[i] << 32) | sh.busy[i];
            acc.tmin = min(acc.tmin, sh.busy[i]);
        } else {
            snap0[sl] = NONE64;
        }
    }
    __syncthreads();
    const uint32_t ns = sh.n_send;
    if (ns) {
        if (tid == 0) sh.send_base = (uint32_t)atomicAdd(&ly.ctl->n_log, (unsigned long long)ns);
        __syncthreads();
        const unsigned long long b0 = sh.send_base;
        for (uint32_t q = tid; q < ns; q += NT) {
            const unsigned long long pos = b0 + q;
            if (pos < ly.ctl->max_sends) {
                ly.skey[0][pos] = ((uint64_t)sh.snd_t[q] << 32) | sh.snd_link[q];
                ly.sval[0][pos] = sh.snd_rank[q];
            } else {
                window_error(ly.ctl, k, ST_ENOMEM, 0, 0, 0);
            }
        }
        if (tid == 0) sent += ns;
    }
    __syncthreads();
}

__global__ void __launch_bounds__(NT) k_match(Layout ly, Sizes sz)
{
    __shared__ Shared sh;
    Control *ctl = ly.ctl;
    if (__hip_atomic_load(&ctl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    const uint32_t tid = threadIdx.x;
    const unsigned long long max_windows = ctl->needs_total + 2ull;
    Acc acc = {NONE32, 0u, 0u, 0ull};
    unsigned long long rounds = 0;
    uint32_t t0 = 0;
    unsigned long long k = 0;
    if (ctl->needs_total == 0) {
        if (blockIdx.x == 0 && tid == 0) ctl->windows = 0;
        return;
    }
    unsigned long long remaining = ctl->needs_total;
    for (;; k++) {
        const uint64_t t1 = (uint64_t)t0 + sz.tmin;
        if (blockIdx.x == 0 && tid == 0) {
            ctl->win_t0[(k + 2) % 3] = NONE32;
            ctl->win_sent[(k + 1) % 3] = 0;
            ctl->win_err[(k + 1) % 3] = 0;
        }
        acc.tmin = NONE32;
        unsigned long long sent = 0;
        for (uint32_t d = blockIdx.x; d < sz.D; d += gridDim.x)
            process_destination(ly, sz, sh, d, (uint32_t)k, t0, t1, acc, rounds, sent);
        const uint32_t bmin = block_min(acc.tmin, sh);
        if (tid == 0) {
            if (bmin != NONE32) atomicMin(&ctl->win_t0[(k + 1) % 3], bmin);
            if (sent) atomicAdd(&ctl->win_sent[k % 3], sent);
        }
        if (!grid_barrier(ctl, sh)) break;
        const uint32_t err = __hip_atomic_load(&ctl->win_err[k % 3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned long long done =
            __hip_atomic_load(&ctl->win_sent[k % 3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t tn = __hip_atomic_load(&ctl->win_t0[(k + 1) % 3], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        remaining -= done;
        if (err || remaining == 0) break;
        if (tn == NONE32) {
            record_error(ctl, ST_EDEADLOCK, (uint32_t)remaining, 0, 0);
            break;
        }
        if (k + 1 >= max_windows) {
            record_error(ctl, ST_EINTERNAL, 1, 0, 0);
            break;
        }
        t0 = tn;
    }
    if (blockIdx.x == 0 && tid == 0) ctl->needs_remaining = remaining;
    // block totals
    uint32_t c = acc.cstar;
    for (int off = 32; off; off >>= 1) c = max(c, (uint32_t)__shfl_xor((int)c, off));
    uint32_t cl = acc.clashes;
    for (int off = 32; off; off >>= 1) cl += (uint32_t)__shfl_xor((int)cl, off);
    if ((tid & 63) == 0) {
        atomicMax(&ctl->cstar, c);
        if (cl) atomicAdd(&ctl->clashes, (unsigned long long)cl);
        if (acc.words) atomicAdd(&ctl->scan_words, (unsigned long long)acc.words);
    }
    if (tid == 0) {
        if (rounds) atomicAdd(&ctl->rounds, rounds);
        if (blockIdx.x == 0) ctl->windows = k + 1;
    }
}

}  // namespace

int match_max_grid(int device)
{
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_match, NT, 0) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return 0;
    return per_cu * cus;
}

hipError_t launch_match(const Layout &ly, const Sizes &sz, hipStream_t st, int grid)
{
    Layout l = ly;
    Sizes s = sz;
    void *args[] = {&l, &s};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k_match), dim3(grid), dim3(NT), args, 0, st);
}

}  // namespace pccl
