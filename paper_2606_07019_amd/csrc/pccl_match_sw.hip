// Matching kernel for networks with explicit switch nodes (Sec. 4.7
// "Modeling Switches"): a switch with a finite buffer takes a new chunk only
// while fewer chunks than its capacity are buffered there, and a switch
// without multicast keeps at most one copy of a chunk in flight on its
// out-links.
//
// The clash groups of these rules reach across destinations: every out-link
// of a unicast switch competes for the same copy, and a limited switch's
// buffer empties as its out-neighbours receive their chunks.  So ownership
// moves from one destination per wavefront to one *switch group* per
// workgroup: a unicast switch's out-neighbours, and a limited switch with its
// out-neighbours, belong to one group (closed under both rules on the host),
// and every other device is a group of its own.  A group's links, link state,
// per-round picks and buffer places live in LDS for the window; its
// destinations' event times are merged and each event runs the round loop of
// the event-stepped matching (pick, clash on (destination, chunk), clash on
// (unicast switch, chunk), free buffer places, commit) with workgroup barriers
// between the stages.  Thread i owns group link i; the picks themselves stay
// inside each wavefront (row scans shared out among its lanes), and hashed
// marks let a pick alone in its clash slot win without comparisons.
//
// When no buffer limit binds, the no-multicast rule can act only if two
// out-neighbours of one unicast switch need the same chunk; k_unicast_check
// finds out after the setup, and this kernel then runs only if they do (the
// plain kernel, queued next to it, runs otherwise).
//
// Groups interact only through chunk arrivals, which take at least the
// smallest link time, so the windows [t0, t0 + Tmin) of the plain matcher
// carry over, with one grid barrier per window: every group reads the
// transfers in flight at t0 (published by their owners at the end of the
// previous window, in one of two alternating planes), folds the transfers
// into its own destinations that end inside the window into their holds
// rows at once, and matches its events against the rows plus the window's
// arrival list; a row chunk whose arrival in the window comes after the
// event is skipped, so the early fold never shows a chunk before its time.
// The barrier at the window's end publishes the next window's entries and
// finds the next event time.
#include "pccl_internal.h"

namespace pccl {
namespace {

constexpr uint32_t ST = SW_THREADS;
constexpr uint32_t SWAVES = ST / 64;
constexpr uint32_t SW_SPIN_LIMIT = 1u << 24;
constexpr uint32_t SCAN_STEP = 4;  // row words one link's scan loads at once
// (link, pair) items of the arrival masks a thread reads in one batch of
// need-word loads: the 8,192 items of a 576-link rail-switch group take
// one batch at 768 threads
constexpr uint32_t AMASK_BATCH = 12;
constexpr uint32_t SW_ADM_LIST = SWAVES * 64u / 2u;  // admissions of a round whose deliveries are counted in the commits
constexpr uint32_t SW_ADM_FILTER = 512;               // words of the round's hashed filter of admitted chunks
static_assert(SW_ADM_FILTER * 32u == 1u << 14, "adm_hash yields 14-bit positions");
constexpr uint32_t PEND = 2;       // needed chunks below a link's cursor it keeps as explicit candidates
static_assert(PEND % 2 == 0, "pending candidates fill whole 64-bit snapshot words");
constexpr uint64_t STAG_MASK = 0xFFFull << 52;
constexpr uint32_t SW_FILTER_WORDS = 512;  // 16,384 filter bits, shared by the group's unicast switches
constexpr uint32_t SW_HASH_WORDS = 2048;   // 32,768 two-bit slots per clash table
static_assert(SW_HASH_WORDS * 16u == 1u << 15, "clash_slot yields 15-bit slots");

static_assert(SW_MAX_LINKS <= SW_THREADS, "the pick stage gives link i to thread i");

struct SwShared {
    // per group link: state, static description and per-round scratch
    uint32_t busy[SW_MAX_LINKS], infl[SW_MAX_LINKS], cur[SW_MAX_LINKS], pick[SW_MAX_LINKS];
    uint32_t lsrc[SW_MAX_LINKS], ldst[SW_MAX_LINKS], ltim[SW_MAX_LINKS], llink[SW_MAX_LINKS];
    uint16_t ldl[SW_MAX_LINKS], lsrcj[SW_MAX_LINKS];
    uint8_t luni[SW_MAX_LINKS], ldbuf[SW_MAX_LINKS], lsbuf[SW_MAX_LINKS];
    // a link's pick in this round won: bit 0 its destination's clash, bit 1
    // also its unicast source switch's, bit 2 also a buffer place
    uint8_t winf[SW_MAX_LINKS];
    uint16_t doff[SW_MAX_LINKS + 1];  // links of destination dl: [doff[dl], doff[dl + 1])
    uint16_t poff[SW_MAX_SRC + 1];    // arrival pairs of source j
    uint32_t arr_t[SW_MAX_PAIRS];     // arrival time inside the window, NONE32 if none
    uint32_t arr_c[SW_MAX_PAIRS];     // arriving chunk
    uint64_t amask[SW_MAX_LINKS];     // arrivals (bit q: pair q of the source) the link's destination needs
    uint32_t pend[SW_MAX_LINKS][PEND];  // needed arrivals outside [cur, hi), NONE32 = empty
    uint32_t hi[SW_MAX_LINKS];          // a link's row candidates lie in [cur, hi) (or in pend)
    uint32_t foldc[SW_MAX_LINKS];       // the chunk a link's transfer delivers inside the window, NONE32 if none
    // where a thread's arrival-mask items start (the link, the pair of its
    // source) and the group's item count: static, set with the group state
    uint16_t it_link[SW_THREADS], it_q[SW_THREADS];
    uint32_t it_tot;
    uint16_t uoff[SW_MAX_SW + 1], ulist[SW_MAX_LINKS];
    uint32_t bcap[SW_MAX_SW];
    uint16_t bpoff[SW_MAX_SW + 1], booff[SW_MAX_SW + 1];
    uint32_t bout[SW_MAX_LINKS];
    uint32_t pc[SW_MAX_POOL], pn[SW_MAX_POOL], occ[SW_MAX_SW];
    // chunks each unicast switch of the group may have in flight (a hashed
    // bit set per switch, a superset: a hit is checked against the links)
    uint32_t filt[SW_FILTER_WORDS];
    // per wave: its links that scan their row in this pick round, in lane order
    uint8_t wsl[SWAVES][64];
    // per unicast switch: its out-links that won their destination's clash
    // in this pick round ([uoff[u], uoff[u] + ucnt[u]) of uwin)
    uint16_t uwin[SW_MAX_LINKS];
    uint32_t ucnt[SW_MAX_SW];
    // per pick round: hashed (destination, chunk) and (unicast switch,
    // chunk) tables of two-bit "seen once / seen again" marks, so that a pick
    // alone in its slot skips the comparison with its rivals; and one bit per
    // destination that picked (rounds are counted per such destination)
    uint32_t hd[SW_HASH_WORDS], hu[SW_HASH_WORDS], dpk[SW_MAX_LINKS / 32];
    // per pick round (two, alternating): bit 0 a pick lost a clash, bit 1 a
    // free link was held back by a full buffer, bit 2 a buffer place was freed
    uint32_t rflag[2];
    // destinations whose links lie in one wave in (link time, link id) order
    // (the buffer-place order is then a ballot and a bit count)
    uint32_t dord[SW_MAX_LINKS / 32];
    // admissions of a round: their number; switch and chunk of each, with
    // the round's deliveries of that chunk to the switch's out-neighbours;
    // a hashed filter of the admitted chunks (set and cleared by the
    // admitting links within the round)
    uint32_t acount;
    uint8_t adm_b[SW_ADM_LIST];
    uint32_t adm_c[SW_ADM_LIST], adel[SW_ADM_LIST];
    uint32_t admf[SW_ADM_FILTER];
    // next send-log slot of each destination of the group (its segment)
    unsigned long long lcur[SW_MAX_LINKS];
    uint32_t red[SWAVES];
    // per wave, at the window barrier: earliest transfer end, transfers
    // committed, error flag (reduced by the thread that publishes the slot)
    uint32_t xr_t[SWAVES], xr_s[SWAVES], xr_e[SWAVES];
    // word positions the workgroup's scans passed (whole run)
    unsigned long long st_words;
    uint32_t x_tmin, x_err, x_ok;
    unsigned long long x_sent;
};

struct SwGroup {
    uint32_t nL, lbase, nD, dbase, nS, sbase, nP, pbase, nU, ubase, ulbase, nB, bbase, bobase, pool_base, pool_n;
};

__device__ inline SwGroup load_group(const SwTab &sw, uint32_t g)
{
    const uint32_t *h = sw.grp + 16ull * g;
    SwGroup x;
    x.nL = h[0];
    x.lbase = h[1];
    x.nD = h[2];
    x.dbase = h[3];
    x.nS = h[4];
    x.sbase = h[5];
    x.nP = h[6];
    x.pbase = h[7];
    x.nU = h[8];
    x.ubase = h[9];
    x.ulbase = h[10];
    x.nB = h[11];
    x.bbase = h[12];
    x.bobase = h[13];
    x.pool_base = h[14];
    x.pool_n = h[15];
    return x;
}

__device__ inline uint8_t small_index(uint32_t v) { return v == NONE32 ? SW_NONE8 : (uint8_t)v; }

// Pending candidates of slot sl when they leave LDS: PEND words in the
// second and third snapshot planes, which this kernel does not use otherwise.
__device__ inline uint64_t pend_index(const Sizes &sz, uint32_t sl)
{
    return (uint64_t)sz.L + (uint64_t)sl * (PEND / 2);
}

__device__ inline bool need_bit(const uint64_t *row, uint32_t c)
{
    const uint64_t w = __hip_atomic_load(&row[c >> 6], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return (w >> (c & 63u)) & 1ull;
}

__device__ inline uint64_t link_key(const SwShared &sh, uint32_t i)
{
    return ((uint64_t)sh.ltim[i] << 32) | sh.llink[i];
}

__device__ inline uint32_t adm_hash(uint32_t c) { return (c * 2654435761u) >> 18; }

// one of the pick round's winners delivers chunk c to group destination dl
// (read after the round's winners are final)
__device__ inline bool delivered_now(const SwShared &sh, uint32_t dl, uint32_t c)
{
    for (uint32_t j = sh.doff[dl], je = sh.doff[dl + 1]; j < je; j++)
        if (sh.pick[j] == c && ((sh.winf[j] >> 2) & 1u)) return true;
    return false;
}

// Cross-lane steps that need no lane-index registers (index arithmetic the
// compiler would hoist out of the loops and spill at this kernel's register
// limit): a lane swizzle exchanges the lanes whose ids differ in bit K
// inside each half of the wave, and the two halves meet through two lane
// reads, whose result is the same on every lane.
template <uint32_t K>
__device__ __forceinline__ uint32_t swz_xor(uint32_t v)
{
    static_assert(K >= 1 && K <= 16 && (K & (K - 1)) == 0, "one lane-id bit inside a half wave");
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, (int)((K << 10) | 0x1Fu));
}

// v itself, opaque to the compiler at this point: address arithmetic
// derived from it is done where it is used instead of being hoisted out of
// the window loop (where, at the register limit, it would be spilled and
// reloaded behind a wait for every load in flight).
__device__ __forceinline__ uint32_t here(uint32_t v)
{
    asm volatile("" : "+v"(v));
    return v;
}

__device__ __forceinline__ uint32_t lane_at(uint32_t v, int l)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

__device__ __forceinline__ uint32_t wave_min(uint32_t v)
{
    v = min(v, swz_xor<16>(v));
    v = min(v, swz_xor<8>(v));
    v = min(v, swz_xor<4>(v));
    v = min(v, swz_xor<2>(v));
    v = min(v, swz_xor<1>(v));
    return min(lane_at(v, 0), lane_at(v, 32));
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v)
{
    v += swz_xor<16>(v);
    v += swz_xor<8>(v);
    v += swz_xor<4>(v);
    v += swz_xor<2>(v);
    v += swz_xor<1>(v);
    return lane_at(v, 0) + lane_at(v, 32);
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v)
{
    v |= swz_xor<16>(v);
    v |= swz_xor<8>(v);
    v |= swz_xor<4>(v);
    v |= swz_xor<2>(v);
    v |= swz_xor<1>(v);
    return lane_at(v, 0) | lane_at(v, 32);
}

static_assert(MAX_MATCH_GRID <= (1u << 13), "the window exchange sums 19-bit counts in 32 bits");

__device__ uint32_t block_min(SwShared &sh, uint32_t v)
{
    v = wave_min(v);
    if ((threadIdx.x & 63) == 0) sh.red[here(threadIdx.x) >> 6] = v;
    __syncthreads();
    uint32_t m = NONE32;
    for (uint32_t w = 0; w < SWAVES; w++) m = min(m, sh.red[w]);
    __syncthreads();
    return m;
}

// Grid barrier with a reduction: every workgroup publishes (tag, error,
// transfers committed, earliest transfer end in flight) in its own 128-byte
// slot; wave 0 polls all slots.  Two slot sets alternate, so a workgroup
// that is already one barrier ahead does not overwrite a slot still read.
// tmin, sent and err are each thread's own: every wave reduces its threads'
// values into an LDS slot before the workgroup barrier, and the thread that
// publishes combines the waves' slots after it.
__device__ bool sw_sync(Control *ctl, uint64_t *xslot, uint32_t gen, uint32_t tmin, uint32_t sent, uint32_t err,
                        SwShared &sh)
{
    const uint32_t nb = gridDim.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t tag = (uint64_t)(gen & 0xFFFu) << 52;
    uint64_t *slot = xslot + (uint64_t)(gen & 1u) * MAX_MATCH_GRID * XSLOT_WORDS;
    tmin = wave_min(tmin);
    sent = wave_sum(sent);
    err = wave_or(err);
    if (lane == 0) {
        const uint32_t wv = here(wave);
        sh.xr_t[wv] = tmin;
        sh.xr_s[wv] = sent;
        sh.xr_e[wv] = err;
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores and atomics are done
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t bt = NONE32, bs = 0, be = 0;
        for (uint32_t w = 0; w < SWAVES; w++) {
            bt = min(bt, sh.xr_t[w]);
            bs += sh.xr_s[w];
            be |= sh.xr_e[w];
        }
        __hip_atomic_store(&slot[(uint64_t)blockIdx.x * XSLOT_WORDS],
                           tag | ((uint64_t)(be ? 1u : 0u) << 51) | ((uint64_t)(bs & 0x7FFFFu) << 32) | bt,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (threadIdx.x < 64) {
        uint32_t spins = 0, ok = 1, tn = NONE32, e = 0;
        unsigned long long s = 0;
        while (true) {
            bool all = true;
            tn = NONE32;
            e = 0;
            s = 0;
            // the abort flag and the slots are loaded together, one round trip
            // per spin (lanes past the last workgroup reread its slot and are
            // ignored, so no load sits under a branch)
            const uint32_t ab = __hip_atomic_load(&ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t b0 = 0; b0 < nb; b0 += 64) {
                const uint64_t a = __hip_atomic_load(&slot[(uint64_t)min(b0 + lane, nb - 1u) * XSLOT_WORDS],
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (b0 + lane >= nb) continue;
                if ((a & STAG_MASK) != tag) all = false;
                tn = min(tn, (uint32_t)a);
                e |= (uint32_t)(a >> 51) & 1u;
                s += (a >> 32) & 0x7FFFFull;
            }
            if (__ballot(!all) == 0) break;
            if (ab) {
                ok = 0;
                break;
            }
            if (++spins > SW_SPIN_LIMIT) {
                if (lane == 0) atomicExch(&ctl->abort, 1u);
                ok = 0;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        // acquire: drop cached lines that other workgroups wrote
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        // (a slot's count has 19 bits and there are at most MAX_MATCH_GRID
        // slots: the sum fits in 32 bits)
        tn = wave_min(tn);
        e = wave_or(e);
        const uint32_t s32 = wave_sum((uint32_t)s);
        if (lane == 0) {
            sh.x_tmin = tn;
            sh.x_err = e;
            sh.x_sent = s32;
            sh.x_ok = ok;
        }
    }
    __syncthreads();
    return sh.x_ok != 0;
}

__device__ void load_group_state(const Layout &ly, const Sizes &sz, const SwGroup &gp, SwShared &sh)
{
    const SwTab &sw = ly.sw;
    const uint32_t tid = threadIdx.x;
    for (uint32_t i = tid; i < gp.nL; i += ST) {
        const uint32_t x = gp.lbase + i, sl = sw.lk_slot[x], l = ly.slot_link[sl];
        sh.llink[i] = l;
        sh.lsrc[i] = ly.lsrc[l];
        sh.ldst[i] = ly.ldst[l];
        sh.ltim[i] = ly.slot_time[sl];
        sh.ldl[i] = (uint16_t)sw.lk_dl[x];
        sh.lsrcj[i] = (uint16_t)sw.lk_srcj[x];
        sh.luni[i] = small_index(sw.lk_uni[x]);
        sh.ldbuf[i] = small_index(sw.lk_dbuf[x]);
        sh.lsbuf[i] = small_index(sw.lk_sbuf[x]);
        sh.busy[i] = ly.busy[sl];
        sh.infl[i] = ly.infl[sl];
        sh.cur[i] = ly.cur[sl];
        sh.hi[i] = (uint32_t)(sz.W * 64) - ly.lflags[sl];  // stored as the distance to the row end
        const uint32_t *pg = reinterpret_cast<const uint32_t *>(ly.snap + pend_index(sz, sl));
#pragma unroll
        for (uint32_t e = 0; e < PEND; e++) sh.pend[i][e] = pg[e];
    }
    for (uint32_t x = tid; x <= gp.nD; x += ST) sh.doff[x] = (uint16_t)sw.d_off[gp.dbase + x];
    for (uint32_t x = tid; x <= gp.nS; x += ST) sh.poff[x] = (uint16_t)sw.s_poff[gp.sbase + x];
    for (uint32_t x = tid; x <= gp.nU; x += ST) sh.uoff[x] = (uint16_t)sw.u_off[gp.ubase + x];
    for (uint32_t x = tid; x <= gp.nB; x += ST) {
        sh.bpoff[x] = (uint16_t)sw.b_poff[gp.bbase + x];
        sh.booff[x] = (uint16_t)sw.b_ooff[gp.bbase + x];
        if (x < gp.nB) {
            sh.bcap[x] = sw.b_cap[gp.bbase + x];
            sh.occ[x] = sw.occ[gp.bbase + x];
        }
    }
    for (uint32_t x = tid; x < gp.pool_n; x += ST) {
        sh.pc[x] = sw.pool_c[gp.pool_base + x];
        sh.pn[x] = sw.pool_n[gp.pool_base + x];
    }
    __syncthreads();
    // list lengths are known once the offsets are in LDS
    const uint32_t nul = gp.nU ? sh.uoff[gp.nU] : 0u;
    for (uint32_t x = tid; x < nul; x += ST) sh.ulist[x] = (uint16_t)sw.u_list[gp.ulbase + x];
    const uint32_t nbo = gp.nB ? sh.booff[gp.nB] : 0u;
    for (uint32_t x = tid; x < nbo; x += ST) sh.bout[x] = sw.b_out[gp.bobase + x];
    for (uint32_t x = tid; x < gp.nD; x += ST)
        if (sh.doff[x] < sh.doff[x + 1]) sh.lcur[x] = ly.dest_log[sh.ldst[sh.doff[x]]];
    // (a wave per 64 destinations, one flag word per 32)
    for (uint32_t x0 = 0; x0 < gp.nD; x0 += ST) {
        const uint32_t x = x0 + tid;
        bool ok = false;
        if (x < gp.nD) {
            const uint32_t a = sh.doff[x], e = sh.doff[x + 1];
            ok = e > a && (a >> 6) == ((e - 1u) >> 6);
            for (uint32_t j = a; ok && j + 1 < e; j++) ok = link_key(sh, j) < link_key(sh, j + 1);
        }
        const uint64_t m = __ballot(ok);
        if ((tid & 63u) == 0 && x < gp.nD) {
            sh.dord[x >> 5] = (uint32_t)m;
            if (x + 32 < gp.nD) sh.dord[(x >> 5) + 1] = (uint32_t)(m >> 32);
        }
    }
    for (uint32_t i = tid; i < gp.nL; i += ST) sh.amask[i] = 0ull;
    // the arrival-mask items: link i's are the pairs of its source; per link
    // its first item (a block prefix, kept in `pick`, which the rounds
    // overwrite), then per thread the link holding its first item (the last
    // link whose first item is at or below it; the walk steps past links
    // without pairs)
    {
        const uint32_t lane = tid & 63u, wave = tid >> 6;
        const uint32_t np_me =
            tid < gp.nL ? (uint32_t)(sh.poff[sh.lsrcj[tid] + 1] - sh.poff[sh.lsrcj[tid]]) : 0u;
        // inclusive prefix over the wave, one lane-id bit per step: `blk`
        // is the sum of the lane's aligned block of 2^k lanes, `inc` its
        // prefix inside the block
        uint32_t inc = np_me, blk = np_me;
        {
            uint32_t o;
            o = swz_xor<1>(blk);
            inc += (lane & 1u) ? o : 0u;
            blk += o;
            o = swz_xor<2>(blk);
            inc += (lane & 2u) ? o : 0u;
            blk += o;
            o = swz_xor<4>(blk);
            inc += (lane & 4u) ? o : 0u;
            blk += o;
            o = swz_xor<8>(blk);
            inc += (lane & 8u) ? o : 0u;
            blk += o;
            o = swz_xor<16>(blk);
            inc += (lane & 16u) ? o : 0u;
            blk += o;
            // (the lane read runs on every lane, outside the select)
            const uint32_t lo = lane_at(blk, 0);
            inc += (lane & 32u) ? lo : 0u;
        }
        if (lane == 63) sh.red[here(wave)] = inc;
        __syncthreads();
        uint32_t below = 0, tot = 0;
        for (uint32_t w = 0; w < SWAVES; w++) {
            const uint32_t r = sh.red[w];
            if (w < wave) below += r;
            tot += r;
        }
        if (tid < gp.nL) sh.pick[tid] = below + inc - np_me;
        if (tid == 0) sh.it_tot = tot;
        __syncthreads();
        const uint32_t x = tid * ((tot + ST - 1) / ST);
        uint32_t lo = 0;
        if (x < tot) {
            uint32_t hi2 = gp.nL;
            while (hi2 - lo > 1) {
                const uint32_t m = (lo + hi2) >> 1;
                if (sh.pick[m] <= x) lo = m;
                else hi2 = m;
            }
        }
        sh.it_link[tid] = (uint16_t)lo;
        sh.it_q[tid] = (uint16_t)(x < tot ? x - sh.pick[lo] : 0u);
    }
}

// A unicast switch keeps one copy of a chunk in flight: is chunk c in flight
// on one of switch u's out-links at time t?
__device__ inline bool sending(const SwShared &sh, uint32_t u, uint32_t c, uint32_t t)
{
    for (uint32_t q = sh.uoff[u]; q < sh.uoff[u + 1]; q++) {
        const uint32_t j = sh.ulist[q];
        if (sh.busy[j] > t && sh.infl[j] == c) return true;
    }
    return false;
}

__device__ inline void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The sending filter: SW_FILTER_WORDS * 32 bits split evenly over the
// group's unicast switches (a power of two each, at least 256 with the
// group limit of 64 switches); chunk c of switch u sets one hashed bit.
__device__ inline uint32_t filter_log2(uint32_t n_uni)
{
    const uint32_t per = (SW_FILTER_WORDS * 32u) / max(n_uni, 1u);
    return 31u - (uint32_t)__builtin_clz(per);
}

__device__ inline uint32_t filter_bit(uint32_t u, uint32_t c, uint32_t fl)
{
    return (u << fl) + ((c * 2654435761u) >> (32u - fl));
}

// Is chunk c in flight on an out-link of unicast switch u at time t?  The
// filter answers "no" for most chunks without walking the links.
__device__ inline bool sent_by(const SwShared &sh, uint32_t u, uint32_t c, uint32_t t, uint32_t fl)
{
    const uint32_t b = filter_bit(u, c, fl);
    return ((sh.filt[b >> 5] >> (b & 31u)) & 1u) && sending(sh, u, c, t);
}

// Slot of (owner, chunk) in a clash table, and its marks: the first insert
// sets bit 0 of the slot, any later one bit 1.  A slot whose bit 1 is clear
// after all inserts holds one pick only.
__device__ inline uint32_t clash_slot(uint32_t owner, uint32_t c)
{
    return ((c ^ (owner * 0x9E3779B9u)) * 2654435761u) >> 17;  // 15 bits
}

__device__ inline void clash_mark(uint32_t *tab, uint32_t slot)
{
    const uint32_t b = 1u << ((slot & 15u) * 2u);
    if (atomicOr(&tab[slot >> 4], b) & b) atomicOr(&tab[slot >> 4], b << 1);
}

__device__ inline bool clash_alone(const uint32_t *tab, uint32_t slot)
{
    return !((tab[slot >> 4] >> ((slot & 15u) * 2u + 1u)) & 1u);
}

// Chunk c, found in the holds row of link i's source, reaches the source
// only after t: each group folds the transfers that end inside a window
// into its destinations' rows when the window opens, so a row can show a
// chunk before its arrival time.  Such a chunk is one of the window's
// arrivals at the source that the link's destination needed at the window
// start, so it is listed in the link's arrival mask, with its time.
__device__ inline bool arrives_later(const SwShared &sh, uint32_t i, uint32_t c, uint32_t t)
{
    const uint32_t base = sh.poff[sh.lsrcj[i]];
    for (uint64_t y = sh.amask[i]; y; y &= y - 1) {
        const uint32_t p = base + (uint32_t)__builtin_ctzll(y);
        if (sh.arr_c[p] == c && sh.arr_t[p] > t) return true;
    }
    return false;
}

// Bits of word w (chunks 64 w .. 64 w + 63) that lie in [lo, hi).
__device__ inline uint64_t range_bits(uint64_t w, uint32_t lo, uint32_t hi)
{
    const uint64_t b0 = w * 64;
    uint64_t m = ~0ull;
    if (b0 + 64 <= lo || b0 >= hi) return 0ull;
    if (b0 < lo) m &= ~0ull << (lo - b0);
    if (b0 + 64 > hi) m &= ~0ull >> (b0 + 64 - hi);
    return m;
}

// The pick of free link i at event t (the BFS step: the first chunk in
// priority order that the source holds and the destination still needs),
// skipping chunks its unicast source switch is already sending.  Candidates
// come from three places: the source's holds row as of the window start,
// scanned from the link's cursor (no such chunk lies below it); earlier
// arrivals kept below the cursor; and chunks arriving at the source inside
// the window up to t.  The needs words are read through the caches: only
// this workgroup clears bits of its destinations' rows and nothing sets them
// while matching, so a cached word can only show a chunk as still needed.
// The lowest candidate is confirmed with one coherent load; a stale one is
// dropped where it came from and the pick repeats.  (One thread per link,
// serial: the pick stage below shares the row scans out among the lanes of
// a wave and calls this only when its candidate turns out stale.)
__device__ __attribute__((noinline)) uint32_t pick_link(const Layout &ly, const Sizes &sz, SwShared &sh, uint32_t i, uint32_t t,
                              unsigned long long &words)
{
    const uint64_t *hs = ly.holds + (uint64_t)sh.lsrc[i] * sz.Wp;
    const uint64_t *nd = ly.needs + (uint64_t)sh.ldst[i] * sz.Wp;
    const uint32_t u = sh.luni[i] == SW_NONE8 ? NONE32 : sh.luni[i];
    const uint32_t base = sh.poff[sh.lsrcj[i]];
    const uint32_t hi = sh.hi[i];
    const uint64_t wend = min<uint64_t>(sz.W, ((uint64_t)hi + 63) >> 6);
    uint32_t skip = 0;  // row hits below this were found delivered in this call
    for (;;) {
        // row: the first cached hit at or above the cursor (the new cursor)
        // and the first one from `skip` on that the source switch is not
        // sending (the row candidate)
        const uint32_t cu = sh.cur[i];
        uint32_t row = NONE32, first = NONE32;
        bool done = false;
        for (uint64_t w0 = cu >> 6; w0 < wend && !done; w0 += SCAN_STEP) {
            // all loads of a step are issued before any is used: a load past
            // the range rereads its last word and is masked out (a load under
            // a branch would make the compiler wait for it where the branches
            // join)
            uint64_t x[SCAN_STEP];
#pragma unroll
            for (uint32_t k = 0; k < SCAN_STEP; k++) {
                const uint64_t w = min<uint64_t>(w0 + k, wend - 1);
                x[k] = hs[w] & nd[w];
            }
#pragma unroll
            for (uint32_t k = 1; k < SCAN_STEP; k++)
                if (w0 + k >= wend) x[k] = 0ull;
            x[0] &= NONE64 << (w0 == (cu >> 6) ? (cu & 63u) : 0u);
            words += min<uint64_t>(SCAN_STEP, wend - w0);
#pragma unroll
            for (uint32_t k = 0; k < SCAN_STEP; k++) {
                for (uint64_t y = done ? 0ull : x[k]; y; y &= y - 1) {
                    const uint32_t c = (uint32_t)((w0 + k) * 64 + (uint64_t)__builtin_ctzll(y));
                    if (c >= hi) {
                        done = true;
                        break;
                    }
                    if (first == NONE32) first = c;
                    if (c >= skip && (u == NONE32 || !sending(sh, u, c, t)) && !arrives_later(sh, i, c, t)) {
                        row = c;
                        done = true;
                        break;
                    }
                }
            }
        }
        sh.cur[i] = first == NONE32 ? max(cu, hi) : first;
        uint32_t best = row, from = 0, slot = 0;
        // earlier arrivals kept below the cursor (their needs words loaded
        // together, word 0 for an empty entry)
        uint64_t pw[PEND];
#pragma unroll
        for (uint32_t e = 0; e < PEND; e++) {
            const uint32_t c = sh.pend[i][e];
            pw[e] = nd[(c == NONE32 ? 0u : c) >> 6];
        }
#pragma unroll
        for (uint32_t e = 0; e < PEND; e++) {
            const uint32_t c = sh.pend[i][e];
            if (c == NONE32 || c >= best) continue;
            if (!((pw[e] >> (c & 63u)) & 1ull)) {
                sh.pend[i][e] = NONE32;
                continue;
            }
            if (u != NONE32 && sending(sh, u, c, t)) continue;
            best = c;
            from = 1;
            slot = e;
        }
        // arrivals up to t that the destination may still need
        for (uint64_t y = sh.amask[i]; y; y &= y - 1) {
            const uint32_t q = (uint32_t)__builtin_ctzll(y), p = base + q, c = sh.arr_c[p];
            if (sh.arr_t[p] > t || c >= best) continue;
            if (u != NONE32 && sending(sh, u, c, t)) continue;
            best = c;
            from = 2;
            slot = q;
        }
        if (best == NONE32 || need_bit(nd, best)) return best;
        // delivered since its word was cached: drop it and pick again
        if (from == 0) {
            if (best == first) sh.cur[i] = best + 1;
            skip = best + 1;
        } else if (from == 1) {
            sh.pend[i][slot] = NONE32;
        } else {
            sh.amask[i] &= ~(1ull << slot);
        }
    }
}

struct SwAcc {
    uint32_t tmin, cstar, err, sent;
    unsigned long long rounds, clashes, words;
};

// A window of one group: its events inside [t0, t1), in time order, each
// with its round loop.  snap_rd holds the transfers in flight when the
// window opens (published at the end of the previous one, indexed by group
// link position); the group publishes its own for the next window in
// snap_wr at the end.
__device__ void match_group(const Layout &ly, const Sizes &sz, const SwGroup &gp, SwShared &sh, uint32_t t0,
                            uint64_t t1, bool first_window, bool resident, SwAcc &acc, const uint64_t *snap_rd,
                            uint64_t *snap_wr)
{
    const uint32_t tid = threadIdx.x;
    // a workgroup with one group keeps its tables and state in LDS
    if (!resident || first_window) load_group_state(ly, sz, gp, sh);
    // the transfers into the group's destinations that end inside the
    // window: their chunks join the destinations' holds rows during the
    // window (issued at its end, next to the published entries, so that no
    // wait for a load in between waits for them too); a reader skips a row
    // chunk whose arrival in this window comes after its event (see
    // arrives_later), and the window exchange makes them visible
    for (uint32_t i = tid; i < gp.nL; i += ST) {
        const uint32_t b = sh.busy[i], c = sh.infl[i];
        sh.foldc[i] = (c != NONE32 && b >= t0 && (uint64_t)b < t1) ? c : NONE32;
    }
    const uint32_t fl = filter_log2(gp.nU);
    // the sending filter is built once per window, from the transfers in
    // flight on the unicast switches' out-links at t0 (a superset at every
    // later event of the window: a set bit only costs the exact check), and
    // commits add theirs as they happen; cleared here, filled below
    const uint32_t nfw = gp.nU ? (gp.nU << fl) >> 5 : 0u;
    for (uint32_t x = tid; x < nfw; x += ST) sh.filt[x] = 0u;
    // arrivals at the group's sources inside the window, from the entries
    // published at t0 (the source's in-links, pair p of source j): eight
    // pairs per thread, so one pass covers a group's 8,192 pairs with two
    // dependent round trips (slot indices, then the entries)
    static_assert(SW_MAX_PAIRS <= 8u * ST, "one pass of eight pairs per thread");
    if (gp.nP) {
        const uint32_t tp = here(tid);
        uint32_t sl[8];
        uint64_t e[8];
#pragma unroll
        for (uint32_t k = 0; k < 8; k++) sl[k] = ly.sw.p_slot[gp.pbase + min(tp + k * ST, gp.nP - 1u)];
#pragma unroll
        for (uint32_t k = 0; k < 8; k++) e[k] = snap_rd[sl[k]];
#pragma unroll
        for (uint32_t k = 0; k < 8; k++) {
            const uint32_t p = tp + k * ST, b = (uint32_t)e[k];
            if (p >= gp.nP) continue;
            const bool in = e[k] != NONE64 && b >= t0 && (uint64_t)b < t1;
            sh.arr_t[p] = in ? b : NONE32;
            sh.arr_c[p] = (uint32_t)(e[k] >> 32);
        }
    }
    __syncthreads();
    // which arrivals each link's destination may still need: the (link,
    // pair) items of all links, spread evenly over the workgroup's threads
    // (each thread's first item was found with the group state); each thread
    // loads the needs words of its items AMASK_BATCH at a time, all in
    // flight together, through the caches (a superset: picks confirm each
    // candidate).  The masks start empty (cleared where the last window
    // used them last).
    {
        const uint32_t tot = sh.it_tot, per = (tot + ST - 1) / ST;
        uint32_t x = tid * per;
        const uint32_t xe = min(x + per, tot);
        if (x < xe) {
            uint32_t i = sh.it_link[tid], q = sh.it_q[tid];
            uint32_t p0 = sh.poff[sh.lsrcj[i]], np = sh.poff[sh.lsrcj[i] + 1] - p0;
            while (x < xe) {
                uint32_t li[AMASK_BATCH], qb[AMASK_BATCH], c[AMASK_BATCH];
                bool v[AMASK_BATCH];
#pragma unroll
                for (uint32_t k = 0; k < AMASK_BATCH; k++) {
                    while (q >= np && i + 1 < gp.nL) {
                        q -= np;
                        i++;
                        p0 = sh.poff[sh.lsrcj[i]];
                        np = sh.poff[sh.lsrcj[i] + 1] - p0;
                    }
                    v[k] = x < xe && q < np && sh.arr_t[p0 + min(q, np - 1u)] != NONE32;
                    li[k] = i;
                    qb[k] = q;
                    c[k] = v[k] ? sh.arr_c[p0 + q] : 0u;
                    x++;
                    q++;
                }
                // unconditional loads (row 0, word 0 for an item without an arrival)
                uint64_t nw[AMASK_BATCH];
#pragma unroll
                for (uint32_t k = 0; k < AMASK_BATCH; k++)
                    nw[k] = ly.needs[(uint64_t)(v[k] ? sh.ldst[li[k]] : 0u) * sz.Wp + (c[k] >> 6)];
#pragma unroll
                for (uint32_t k = 0; k < AMASK_BATCH; k++)
                    if (v[k] && ((nw[k] >> (c[k] & 63u)) & 1ull))
                        atomicOr((unsigned long long *)&sh.amask[li[k]], 1ull << qb[k]);
            }
        }
        if (gp.nU)
            for (uint32_t i = tid; i < gp.nL; i += ST) {
                const uint32_t u = sh.luni[i];
                if (u != SW_NONE8 && sh.infl[i] != NONE32 && (uint64_t)sh.busy[i] > (uint64_t)t0) {
                    const uint32_t b = filter_bit(u, sh.infl[i], fl);
                    atomicOr(&sh.filt[b >> 5], 1u << (b & 31u));
                }
            }
        // the round tables start empty
        for (uint32_t x = tid; x < SW_HASH_WORDS; x += ST) {
            sh.hd[x] = 0u;
            sh.hu[x] = 0u;
        }
        for (uint32_t x = tid; x < SW_MAX_LINKS / 32; x += ST) sh.dpk[x] = 0u;
        for (uint32_t x = tid; x < SW_ADM_FILTER; x += ST) sh.admf[x] = 0u;
        if (tid < 2) sh.rflag[tid] = 0u;
        __syncthreads();
    }
    uint32_t par = 0;  // this round's rflag word
    int64_t t_prev = first_window ? -1 : (int64_t)t0 - 1;
    for (;;) {
        // next event of the group: a transfer into it ends, or a chunk
        // arrives at one of its sources (time 0 opens the first window)
        uint32_t m = (first_window && t_prev < 0) ? 0u : NONE32;
        for (uint32_t i = tid; i < gp.nL; i += ST) {
            const uint32_t b = sh.busy[i];
            if (sh.infl[i] != NONE32 && (int64_t)b > t_prev && (uint64_t)b < t1) m = min(m, b);
        }
        for (uint32_t p = tid; p < gp.nP; p += ST) {
            const uint32_t a = sh.arr_t[p];
            if (a != NONE32 && (int64_t)a > t_prev) m = min(m, a);
        }
        const uint32_t t = block_min(sh, m);
        if (t == NONE32) break;
        for (;;) {
            // a pick into a limited switch: how many of the switch's
            // out-links lead to a device that needs the chunk, before this
            // round's commits (loaded with the pick, used if it is admitted)
            uint32_t acl = 0;
            // picks of the free links (a full buffer admits nothing), in three
            // steps inside each wave: every free link's lowest explicit
            // candidate (pending or arrived); the row scans below it, shared
            // out among the wave's lanes; the lower of the two, confirmed
            // with one coherent load (thread tid owns link tid)
            {
                const uint32_t i = tid, lane = tid & 63u, wave = tid >> 6;
                bool free = false;
                uint32_t u = NONE32, bxv = NONE32, cu = 0, lim = 0;
                const uint64_t *nd = ly.needs;
                if (i < gp.nL && sh.busy[i] <= t) {
                    const uint32_t b = sh.ldbuf[i];
                    free = b == SW_NONE8 || sh.occ[b] < sh.bcap[b];
                    if (!free) atomicOr(&sh.rflag[par], 2u);
                }
                if (free) {
                    nd = ly.needs + (uint64_t)sh.ldst[i] * sz.Wp;
                    u = sh.luni[i] == SW_NONE8 ? NONE32 : sh.luni[i];
                    // earlier arrivals kept below the cursor (needs words
                    // loaded together, word 0 for an empty entry)
                    uint64_t pw[PEND];
#pragma unroll
                    for (uint32_t e = 0; e < PEND; e++) {
                        const uint32_t c = sh.pend[i][e];
                        pw[e] = nd[(c == NONE32 ? 0u : c) >> 6];
                    }
#pragma unroll
                    for (uint32_t e = 0; e < PEND; e++) {
                        const uint32_t c = sh.pend[i][e];
                        if (c == NONE32 || c >= bxv) continue;
                        if (!((pw[e] >> (c & 63u)) & 1ull)) {
                            sh.pend[i][e] = NONE32;
                            continue;
                        }
                        if (u != NONE32 && sent_by(sh, u, c, t, fl)) continue;
                        bxv = c;
                    }
                    // arrivals up to t that the destination may still need
                    const uint32_t base = sh.poff[sh.lsrcj[i]];
                    for (uint64_t y = sh.amask[i]; y; y &= y - 1) {
                        const uint32_t p = base + (uint32_t)__builtin_ctzll(y), c = sh.arr_c[p];
                        if (sh.arr_t[p] > t || c >= bxv) continue;
                        if (u != NONE32 && sent_by(sh, u, c, t, fl)) continue;
                        bxv = c;
                    }
                    // the row matters below the explicit candidate only
                    cu = sh.cur[i];
                    lim = min(sh.hi[i], bxv);
                }
                const bool scan = free && cu < lim;
                if (__ballot(scan)) {
                    // Steps of G = 64 / next_pow2(k) lanes for each of the k
                    // links still scanning, four words per lane; the lanes are
                    // dealt again before every step, so the few links whose
                    // scan runs long get the whole wave.  A link's position,
                    // first hit (its new cursor) and first hit the source
                    // switch is not sending (its row candidate) stay on the
                    // link's own lane; a min over each lane group gives the
                    // step's result, which the group's first lane hands back.
                    const uint64_t below = (1ull << lane) - 1ull;
                    uint32_t opos = (cu >> 6) & ~3u, ofh = NONE32, orc = NONE32;
                    const uint32_t owl = (uint32_t)(((uint64_t)lim + 63u) >> 6);
                    bool olive = scan;
                    for (;;) {
                        const uint64_t lm = __ballot(olive);
                        if (!lm) break;
                        const uint32_t rank = (uint32_t)__popcll(lm & below);
                        if (olive) sh.wsl[wave][rank] = (uint8_t)lane;
                        wave_sync();
                        const uint32_t ks = (uint32_t)__popcll(lm);
                        const uint32_t lg = ks <= 1u ? 0u : 32u - (uint32_t)__builtin_clz(ks - 1u);
                        const uint32_t G = 64u >> lg, g = lane >> (6u - lg), sub = lane & (G - 1u);
                        const bool act = g < ks;
                        const uint32_t jl = sh.wsl[wave][act ? g : 0u];
                        const uint32_t pj = (uint32_t)__shfl((int)opos, (int)jl);
                        const uint32_t cj = (uint32_t)__shfl((int)cu, (int)jl);
                        const uint32_t lj = (uint32_t)__shfl((int)lim, (int)jl);
                        const uint32_t uj = (uint32_t)__shfl((int)u, (int)jl);
                        const uint32_t ij = (wave << 6) | jl;
                        const uint64_t *hrow = ly.holds + (uint64_t)sh.lsrc[ij] * sz.Wp;
                        const uint64_t *nrow = ly.needs + (uint64_t)sh.ldst[ij] * sz.Wp;
                        const uint64_t wl = ((uint64_t)lj + 63u) >> 6;
                        // loads at a clamped, always valid word pair (rows
                        // have an even number of words), masked after
                        const uint64_t w = (uint64_t)pj + 4ull * sub;
                        const uint64_t wc = min<uint64_t>(w, sz.Wp - 4);
                        const uint4 hv = *reinterpret_cast<const uint4 *>(hrow + wc);
                        const uint4 nv = *reinterpret_cast<const uint4 *>(nrow + wc);
                        const uint4 hv2 = *reinterpret_cast<const uint4 *>(hrow + wc + 2);
                        const uint4 nv2 = *reinterpret_cast<const uint4 *>(nrow + wc + 2);
                        uint32_t lfh = NONE32, lrc = NONE32;
                        if (act && w < wl) {
                            uint64_t a[4];
                            a[0] = ((((uint64_t)hv.y << 32) | hv.x) & (((uint64_t)nv.y << 32) | nv.x)) &
                                   range_bits(w, cj, lj);
                            a[1] = ((((uint64_t)hv.w << 32) | hv.z) & (((uint64_t)nv.w << 32) | nv.z)) &
                                   range_bits(w + 1, cj, lj);
                            a[2] = ((((uint64_t)hv2.y << 32) | hv2.x) & (((uint64_t)nv2.y << 32) | nv2.x)) &
                                   range_bits(w + 2, cj, lj);
                            a[3] = ((((uint64_t)hv2.w << 32) | hv2.z) & (((uint64_t)nv2.w << 32) | nv2.z)) &
                                   range_bits(w + 3, cj, lj);
#pragma unroll
                            for (uint32_t k = 0; k < 4; k++) {
                                for (uint64_t y = lrc == NONE32 ? a[k] : 0ull; y; y &= y - 1) {
                                    const uint32_t c = (uint32_t)((w + k) * 64 + (uint64_t)__builtin_ctzll(y));
                                    if (lfh == NONE32) lfh = c;
                                    if ((uj == NONE32 || !sent_by(sh, uj, c, t, fl)) && !arrives_later(sh, ij, c, t)) {
                                        lrc = c;
                                        break;
                                    }
                                }
                            }
                        }
                        {
                            // word positions of the step, counted by the wave
                            const uint64_t sm = __ballot(act && w < wl);
                            if (lane == 0 && sm) atomicAdd(&sh.st_words, 4ull * (uint64_t)__popcll(sm));
                        }
                        // (G is the same on every lane of the wave)
                        if (G > 1u) {
                            lfh = min(lfh, swz_xor<1>(lfh));
                            lrc = min(lrc, swz_xor<1>(lrc));
                        }
                        if (G > 2u) {
                            lfh = min(lfh, swz_xor<2>(lfh));
                            lrc = min(lrc, swz_xor<2>(lrc));
                        }
                        if (G > 4u) {
                            lfh = min(lfh, swz_xor<4>(lfh));
                            lrc = min(lrc, swz_xor<4>(lrc));
                        }
                        if (G > 8u) {
                            lfh = min(lfh, swz_xor<8>(lfh));
                            lrc = min(lrc, swz_xor<8>(lrc));
                        }
                        if (G > 16u) {
                            lfh = min(lfh, swz_xor<16>(lfh));
                            lrc = min(lrc, swz_xor<16>(lrc));
                        }
                        if (G > 32u) {
                            lfh = min(lane_at(lfh, 0), lane_at(lfh, 32));
                            lrc = min(lane_at(lrc, 0), lane_at(lrc, 32));
                        }
                        // (an owner's group is its rank among the live links)
                        const uint32_t src = (rank * G) & 63u;
                        const uint32_t rfh = (uint32_t)__shfl((int)lfh, (int)src);
                        const uint32_t rrc = (uint32_t)__shfl((int)lrc, (int)src);
                        if (olive) {
                            ofh = min(ofh, rfh);
                            opos += 4u * G;
                            if (rrc != NONE32) {
                                orc = rrc;
                                olive = false;
                            } else if (opos >= owl) {
                                olive = false;
                            }
                        }
                        // (the list is rewritten for the next step)
                        wave_sync();
                    }
                    if (scan) {
                        sh.pick[i] = orc;
                        sh.cur[i] = ofh != NONE32 ? ofh : max(cu, lim);
                    }
                }
                uint32_t pk = NONE32;
                if (free) {
                    pk = min(scan ? sh.pick[i] : NONE32, bxv);
                    // a candidate delivered since its needs word was cached:
                    // the serial pick drops it and finds the next one
                    if (pk != NONE32 && !need_bit(nd, pk)) {
                        // (a local counter: the thread's statistics stay in
                        // registers, out of the call's reach)
                        unsigned long long pw = 0;
                        pk = pick_link(ly, sz, sh, i, t, pw);
                        acc.words += pw;
                    }
                }
                if (i < gp.nU) sh.ucnt[i] = 0u;
                if (i == 0) sh.acount = 0u;
                if (i < gp.nL) sh.pick[i] = pk;
                if (pk != NONE32 && sh.ldbuf[i] != SW_NONE8)
                    acl = __hip_atomic_load(&ly.sw.acnt[(uint64_t)(gp.bbase + sh.ldbuf[i]) * sz.C + pk],
                                            __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (pk != NONE32) {
                    const uint32_t dl = sh.ldl[i];
                    clash_mark(sh.hd, clash_slot(dl, pk));
                    if (!(atomicOr(&sh.dpk[dl >> 5], 1u << (dl & 31u)) & (1u << (dl & 31u)))) acc.rounds++;
                }
            }
            __syncthreads();
            // clash on (destination, chunk): fastest link, then lowest id
            for (uint32_t i = tid; i < gp.nL; i += ST) {
                const uint32_t pk = sh.pick[i];
                uint8_t w = pk != NONE32;
                if (w) {
                    const uint32_t dl = sh.ldl[i];
                    if (!clash_alone(sh.hd, clash_slot(dl, pk))) {
                        const uint64_t key = link_key(sh, i);
                        for (uint32_t j0 = sh.doff[dl], je = sh.doff[dl + 1]; j0 < je; j0 += 4) {
                            uint32_t pj[4];
#pragma unroll
                            for (uint32_t k = 0; k < 4; k++) pj[k] = sh.pick[min(j0 + k, je - 1u)];
#pragma unroll
                            for (uint32_t k = 0; k < 4; k++) {
                                const uint32_t j = j0 + k;
                                if (j < je && j != i && pj[k] == pk && link_key(sh, j) < key) w = 0;
                            }
                        }
                    }
                    const uint32_t u = sh.luni[i];
                    if (w && u != SW_NONE8) {
                        sh.uwin[sh.uoff[u] + atomicAdd(&sh.ucnt[u], 1u)] = (uint16_t)i;
                        clash_mark(sh.hu, clash_slot(u, pk));
                    }
                }
                sh.winf[i] = w;
            }
            __syncthreads();
            // clash on (unicast switch, chunk) among the destination winners
            for (uint32_t i = tid; i < gp.nL; i += ST) {
                uint8_t w = sh.winf[i];
                const uint32_t u = sh.luni[i];
                if (w && u != SW_NONE8 && !clash_alone(sh.hu, clash_slot(u, sh.pick[i]))) {
                    const uint32_t pk = sh.pick[i];
                    const uint64_t key = link_key(sh, i);
                    for (uint32_t q = sh.uoff[u], qe = q + sh.ucnt[u]; q < qe; q++) {
                        const uint32_t j = sh.uwin[q];
                        if (j != i && sh.pick[j] == pk && link_key(sh, j) < key) w = 0;
                    }
                }
                sh.winf[i] = w ? 3u : 0u;
            }
            __syncthreads();
            // free places of a limited switch, in (link time, link id) order
            uint32_t myadm = NONE32;
            {
                const uint32_t i = tid;
                const uint8_t wf = i < gp.nL ? sh.winf[i] : 0u;
                uint32_t w = (wf >> 1) & 1u;
                const uint32_t b = i < gp.nL ? sh.ldbuf[i] : SW_NONE8;
                const uint64_t w2m = __ballot(w != 0u);
                if (w && b != SW_NONE8) {
                    const uint32_t dl = sh.ldl[i];
                    uint32_t ahead = 0;
                    if ((sh.dord[dl >> 5] >> (dl & 31u)) & 1u) {
                        // the destination's winners with a smaller key are its
                        // winners on lower lanes of this wave
                        const uint32_t lo = sh.doff[dl] & 63u, me = i & 63u;
                        ahead = (uint32_t)__popcll(w2m & ((1ull << me) - 1ull) & ~((1ull << lo) - 1ull));
                    } else {
                        const uint64_t key = link_key(sh, i);
                        for (uint32_t j0 = sh.doff[dl], je = sh.doff[dl + 1]; j0 < je; j0 += 4) {
                            uint8_t fj[4];
#pragma unroll
                            for (uint32_t k = 0; k < 4; k++) fj[k] = j0 + k < je ? sh.winf[min(j0 + k, je - 1u)] : 0u;
#pragma unroll
                            for (uint32_t k = 0; k < 4; k++)
                                if (j0 + k != i && ((fj[k] >> 1) & 1u) && link_key(sh, j0 + k) < key) ahead++;
                        }
                    }
                    if (ahead >= sh.bcap[b] - sh.occ[b]) w = 0;
                }
                // (bits 0 and 1, which other links read in this stage, keep their values)
                if (i < gp.nL) sh.winf[i] = (uint8_t)((wf & 3u) | (w << 2));
                if (w && b != SW_NONE8) {
                    const uint32_t pk = sh.pick[i], h = adm_hash(pk);
                    myadm = atomicAdd(&sh.acount, 1u);
                    if (myadm < SW_ADM_LIST) {
                        sh.adm_b[myadm] = (uint8_t)b;
                        sh.adm_c[myadm] = pk;
                        sh.adel[myadm] = 0u;
                    }
                    atomicOr(&sh.admf[h >> 5], 1u << (h & 31u));
                }
            }
            // the counts are read before any commit of this round updates them
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
            __syncthreads();
            // commit: the destination no longer needs the chunk, so neither
            // do the limited switches feeding it on its behalf (and the
            // round's clash tables are cleared for the next round)
            for (uint32_t x = tid; x < SW_HASH_WORDS; x += ST) {
                sh.hd[x] = 0u;
                sh.hu[x] = 0u;
            }
            for (uint32_t x = tid; x < SW_MAX_LINKS / 32; x += ST) sh.dpk[x] = 0u;
            // the next round's flags (last read right after the previous
            // round's final barrier, first set after this round's)
            if (tid == 0) sh.rflag[par ^ 1u] = 0u;
            uint32_t mine = 0;
            for (uint32_t i = tid; i < gp.nL; i += ST) {
                const uint32_t pk = sh.pick[i];
                if (pk == NONE32) continue;
                if (!((sh.winf[i] >> 2) & 1u)) {
                    acc.clashes++;
                    atomicOr(&sh.rflag[par], 1u);
                    continue;
                }
                const uint32_t d = sh.ldst[i];
                __hip_atomic_fetch_and(&ly.needs[(uint64_t)d * sz.Wp + (pk >> 6)], ~(1ull << (pk & 63u)),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                const uint32_t dl = sh.ldl[i];
                if (gp.nB) {
                    for (uint32_t j0 = sh.doff[dl], je = sh.doff[dl + 1]; j0 < je; j0 += 8) {
                        uint8_t bj[8];
#pragma unroll
                        for (uint32_t k = 0; k < 8; k++) bj[k] = j0 + k < je ? sh.lsbuf[min(j0 + k, je - 1u)] : SW_NONE8;
#pragma unroll
                        for (uint32_t k = 0; k < 8; k++) {
                            const uint32_t b = bj[k];
                            if (b == SW_NONE8) continue;
                            // one out-link of b less leads to a device needing
                            // pk (and a delivery of an admission's chunk to
                            // its switch's out-neighbour is counted for it)
                            __hip_atomic_fetch_sub(&ly.sw.acnt[(uint64_t)(gp.bbase + b) * sz.C + pk], 1u,
                                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            const uint32_t h = adm_hash(pk);
                            if ((sh.admf[h >> 5] >> (h & 31u)) & 1u) {
                                const uint32_t na = min(sh.acount, SW_ADM_LIST);
                                for (uint32_t a = 0; a < na; a++)
                                    if (sh.adm_c[a] == pk && sh.adm_b[a] == b) atomicAdd(&sh.adel[a], 1u);
                            }
                            // the place holding pk, four places compared at a time
                            bool done = false;
                            for (uint32_t s0 = sh.bpoff[b], se = sh.bpoff[b + 1]; s0 < se && !done; s0 += 4) {
                                uint32_t cs[4];
#pragma unroll
                                for (uint32_t m = 0; m < 4; m++) cs[m] = sh.pc[min(s0 + m, se - 1u)];
#pragma unroll
                                for (uint32_t m = 0; m < 4; m++) {
                                    const uint32_t s = s0 + m;
                                    if (done || s >= se || cs[m] != pk || sh.pn[s] == 0u) continue;
                                    if (atomicSub(&sh.pn[s], 1u) == 1u) {
                                        atomicSub(&sh.occ[b], 1u);
                                        atomicOr(&sh.rflag[par], 4u);
                                    }
                                    done = true;
                                }
                            }
                        }
                    }
                }
                const uint64_t end = (uint64_t)t + sh.ltim[i];
                if (end > 0xFFFFFFFFull) {
                    record_error(ly.ctl, ST_ERANGE, pk, d, 2);
                    acc.err = 1;
                }
                const uint32_t e32 = end > 0xFFFFFFFFull ? NONE32 - 1u : (uint32_t)end;
                sh.busy[i] = e32;
                sh.infl[i] = pk;
                const uint32_t u = sh.luni[i];
                if (u != SW_NONE8) {
                    const uint32_t fb = filter_bit(u, pk, fl);
                    atomicOr(&sh.filt[fb >> 5], 1u << (fb & 31u));
                }
                acc.cstar = max(acc.cstar, e32);
                const unsigned long long q = atomicAdd(&sh.lcur[dl], 1ull);
                ly.skey[0][q] = ((uint64_t)t << 32) | sh.llink[i];
                ly.sval[0][q] = pk;
                mine++;
            }
            __syncthreads();
            // a limited switch that took a chunk buffers it while an
            // out-link leads to a device that still needs it after this
            // round's commits: the count loaded with the pick less the
            // round's deliveries of the chunk to the switch's out-neighbours
            // (every one of them is a destination of this group), counted by
            // the commits (past the listed admissions, asked here link by
            // link); then the admitting link takes a free place
            if (myadm != NONE32) {
                const uint32_t i = tid, b = sh.ldbuf[i], pk = sh.pick[i], h = adm_hash(pk);
                atomicAnd(&sh.admf[h >> 5], ~(1u << (h & 31u)));
                uint32_t got = 0;
                if (myadm < SW_ADM_LIST) {
                    got = sh.adel[myadm];
                } else {
                    for (uint32_t q = sh.booff[b], qe = sh.booff[b + 1]; q < qe; q++)
                        got += delivered_now(sh, sh.bout[q] >> 16, pk) ? 1u : 0u;
                }
                const uint32_t cnt = acl - got;
                if (cnt)
                    for (uint32_t s = sh.bpoff[b]; s < sh.bpoff[b + 1]; s++)
                        if (atomicCAS(&sh.pn[s], 0u, cnt) == 0u) {
                            sh.pc[s] = pk;
                            atomicAdd(&sh.occ[b], 1u);
                            break;
                        }
            }
            acc.sent += mine;
            // the commits' needs and count updates are done before the next
            // round's picks read them
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
            // another round picks something only for a link that lost a
            // clash, or one a full buffer held back when a place was freed:
            // holds do not change inside an event, needs and free places only
            // shrink otherwise, and chunks in flight only add up
            __syncthreads();
            const uint32_t f = sh.rflag[par];
            par ^= 1u;
            if (!(f & 1u) && (f & 6u) != 6u) break;
        }
        t_prev = t;
    }
    // chunks that arrived at a source inside the window join its holds row
    // at the next window start, possibly outside the region [cur, hi) a
    // link still scans: the link keeps the ones its destination still needs
    // as pending candidates, and only when those are full widens the region
    // to cover them (the others can never be candidates again)
    uint32_t tm = NONE32;
    for (uint32_t i = tid; i < gp.nL; i += ST) {
        const uint64_t *nd = ly.needs + (uint64_t)sh.ldst[i] * sz.Wp;
        const uint32_t base = sh.poff[sh.lsrcj[i]];
        uint32_t c = sh.cur[i], h = sh.hi[i];
        // the region only grows below, so the arrivals outside it now are
        // the only ones whose need is asked: their words are loaded first
        uint64_t out = 0, needed = 0;
        for (uint64_t y = sh.amask[i]; y; y &= y - 1) {
            const uint32_t q = (uint32_t)__builtin_ctzll(y), ac = sh.arr_c[base + q];
            if (!(c <= ac && ac < h)) out |= 1ull << q;
        }
        while (out) {
            uint32_t q[8], ac[8];
#pragma unroll
            for (uint32_t k = 0; k < 8; k++) {
                q[k] = out ? (uint32_t)__builtin_ctzll(out) : 64u;
                out &= out - 1;
                ac[k] = q[k] < 64u ? sh.arr_c[base + q[k]] : 0u;
            }
            uint64_t nw[8];
#pragma unroll
            for (uint32_t k = 0; k < 8; k++)
                nw[k] = __hip_atomic_load(&nd[ac[k] >> 6], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
            for (uint32_t k = 0; k < 8; k++)
                if (q[k] < 64u && ((nw[k] >> (ac[k] & 63u)) & 1ull)) needed |= 1ull << q[k];
        }
        for (uint64_t y = sh.amask[i]; y; y &= y - 1) {
            const uint32_t q = (uint32_t)__builtin_ctzll(y), ac = sh.arr_c[base + q];
            if ((c <= ac && ac < h) || !((needed >> q) & 1ull)) continue;
            uint32_t e = 0;
            while (e < PEND && sh.pend[i][e] != NONE32 && sh.pend[i][e] != ac) e++;
            if (e < PEND) {
                sh.pend[i][e] = ac;
            } else if (c >= h) {
                c = ac;
                h = ac + 1;
            } else {
                c = min(c, ac);
                h = max(h, ac + 1);
            }
        }
        sh.cur[i] = c;
        sh.hi[i] = h;
        sh.amask[i] = 0ull;  // (the next window's masks start empty)
        // the next window's entry: the transfer still in flight at its start
        const bool fl_next = sh.infl[i] != NONE32 && (uint64_t)sh.busy[i] >= t1;
        __hip_atomic_store(&snap_wr[gp.lbase + i], fl_next ? (((uint64_t)sh.infl[i] << 32) | sh.busy[i]) : NONE64,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t fc = sh.foldc[i];
        if (fc != NONE32)
            __hip_atomic_fetch_or(&ly.holds[(uint64_t)sh.ldst[i] * sz.Wp + (fc >> 6)], 1ull << (fc & 63u),
                                  __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (fl_next) tm = min(tm, sh.busy[i]);
        if (!resident) {
            const uint32_t sl = ly.sw.lk_slot[gp.lbase + i];
            ly.cur[sl] = c;
            ly.lflags[sl] = (uint32_t)(sz.W * 64) - h;
            ly.busy[sl] = sh.busy[i];
            ly.infl[sl] = sh.infl[i];
            uint32_t *pg = reinterpret_cast<uint32_t *>(ly.snap + pend_index(sz, sl));
#pragma unroll
            for (uint32_t e = 0; e < PEND; e++) pg[e] = sh.pend[i][e];
        }
    }
    acc.tmin = min(acc.tmin, tm);
    if (!resident) {
        for (uint32_t x = tid; x < gp.nD; x += ST)
            if (sh.doff[x] < sh.doff[x + 1]) ly.dest_log[sh.ldst[sh.doff[x]]] = sh.lcur[x];
        for (uint32_t x = tid; x < gp.pool_n; x += ST) {
            ly.sw.pool_c[gp.pool_base + x] = sh.pc[x];
            ly.sw.pool_n[gp.pool_base + x] = sh.pn[x];
        }
        for (uint32_t x = tid; x < gp.nB; x += ST) ly.sw.occ[gp.bbase + x] = sh.occ[x];
        // (the next group's state replaces this one's in LDS)
        __syncthreads();
    }
}

// Can the no-multicast rule change the schedule?  Only when two
// out-neighbours of one unicast switch need the same chunk (the needs rows as
// set up, relay marks included, over the whole run: needs only shrink).
// Otherwise no two out-links of a unicast switch ever pick the same chunk, so
// the rule never acts and, with no binding buffer limit, the plain matching
// gives the same schedule.  One thread per (unicast switch, row word).
__global__ void __launch_bounds__(256) k_unicast_check(Layout ly, Sizes sz)
{
    if (__hip_atomic_load(&ly.ctl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    const uint32_t u = blockIdx.y;
    const uint64_t x = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    if (x >= sz.W) return;
    const uint32_t q0 = ly.sw.uc_off[u], q1 = ly.sw.uc_off[u + 1];
    uint64_t acc = 0, twice = 0;
    for (uint32_t q = q0; q < q1; q += 8) {
        uint64_t w[8];
#pragma unroll
        for (uint32_t k = 0; k < 8; k++) w[k] = ly.needs[(uint64_t)ly.sw.uc_dst[min(q + k, q1 - 1u)] * sz.Wp + x];
#pragma unroll
        for (uint32_t k = 0; k < 8; k++)
            if (q + k < q1) {
                twice |= acc & w[k];
                acc |= w[k];
            }
    }
    if (twice) atomicOr(&ly.ctl->sw_binds, 1u);
}

__global__ void __launch_bounds__(ST) k_match_sw(Layout ly, Sizes sz)
{
    __shared__ SwShared sh;
    Control *ctl = ly.ctl;
    if (__hip_atomic_load(&ctl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    // queued next to the plain kernel: runs only when the check found that
    // the no-multicast rule can act
    if (sz.sw_gate && !__hip_atomic_load(&ctl->sw_binds, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    const uint32_t tid = threadIdx.x;
    if (ctl->needs_total == 0) {
        if (blockIdx.x == 0 && tid == 0) ctl->windows = 0;
        return;
    }
    const SwTab &sw = ly.sw;
    const uint32_t q0 = sw.blk[blockIdx.x], q1 = sw.blk[blockIdx.x + 1];
    const bool resident = q1 - q0 == 1;
    // empty buffers
    for (uint32_t q = q0; q < q1; q++) {
        const SwGroup gp = load_group(sw, sw.blk_list[q]);
        for (uint32_t x = tid; x < gp.pool_n; x += ST) sw.pool_n[gp.pool_base + x] = 0u;
        for (uint32_t x = tid; x < gp.nB; x += ST) sw.occ[gp.bbase + x] = 0u;
    }
    const unsigned long long max_windows = ctl->needs_total + 2ull;
    unsigned long long remaining = ctl->needs_total;
    SwAcc acc = {NONE32, 0u, 0u, 0u, 0ull, 0ull, 0ull};
    if (tid == 0) sh.st_words = 0ull;
    __syncthreads();
    uint32_t t0 = 0, gen = 0;
    unsigned long long k = 0;
    // two snapshot planes (the first and the third; the second holds the
    // pending candidates of groups that leave LDS), alternating by window
    uint64_t *const plane[2] = {ly.snap, ly.snap + 2ull * sz.L};
    for (;; k++) {
        const uint64_t t1 = (uint64_t)t0 + sz.tmin;
        acc.tmin = NONE32;
        acc.sent = 0;
        for (uint32_t q = q0; q < q1; q++)
            match_group(ly, sz, load_group(sw, sw.blk_list[q]), sh, t0, t1, k == 0, resident, acc, plane[k & 1],
                        plane[(k + 1) & 1]);
        if (!sw_sync(ctl, ly.xslot, ++gen, acc.tmin, acc.sent, acc.err ? 1u : 0u, sh)) break;
        remaining -= sh.x_sent;
        if (sh.x_err || remaining == 0) break;
        if (sh.x_tmin == NONE32) {
            record_error(ctl, ST_EDEADLOCK, (uint32_t)remaining, 0, 0);
            break;
        }
        if (k + 1 >= max_windows) {
            record_error(ctl, ST_EINTERNAL, 1, 0, 0);
            break;
        }
        t0 = sh.x_tmin;
    }
    if (blockIdx.x == 0 && tid == 0) {
        ctl->needs_remaining = remaining;
        ctl->windows = k + 1;
        ctl->n_log = ctl->needs_total - remaining;
    }
    for (int off = 32; off; off >>= 1) {
        acc.cstar = max(acc.cstar, (uint32_t)__shfl_xor(acc.cstar, off));
        acc.rounds += (unsigned long long)__shfl_xor(acc.rounds, off);
        acc.clashes += (unsigned long long)__shfl_xor(acc.clashes, off);
        acc.words += (unsigned long long)__shfl_xor(acc.words, off);
    }
    __syncthreads();
    if (tid == 0 && sh.st_words) atomicAdd(&ctl->scan_words, sh.st_words);
    if ((tid & 63) == 0) {
        atomicMax(&ctl->cstar, acc.cstar);
        if (acc.clashes) atomicAdd(&ctl->clashes, acc.clashes);
        if (acc.words) atomicAdd(&ctl->scan_words, acc.words);
        if (acc.rounds) atomicAdd(&ctl->rounds, acc.rounds);
    }
}

}  // namespace

int match_sw_max_grid(int device)
{
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_match_sw, ST, 0) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return 0;
    return per_cu * cus;
}

hipError_t launch_unicast_check(const Layout &ly, const Sizes &sz, hipStream_t st, uint32_t n_uni)
{
    if (n_uni == 0 || sz.W == 0) return hipSuccess;
    if (n_uni > 65535u) return hipErrorInvalidValue;
    const uint64_t bx = (sz.W + 255) / 256;
    if (bx > 0x7FFFFFFFull) return hipErrorInvalidValue;
    k_unicast_check<<<dim3((uint32_t)bx, n_uni), 256, 0, st>>>(ly, sz);
    return hipGetLastError();
}

hipError_t launch_match_sw(const Layout &ly, const Sizes &sz, hipStream_t st, int grid)
{
    if (grid < 1 || grid > (int)MAX_MATCH_GRID) return hipErrorInvalidValue;
    Layout l = ly;
    Sizes s = sz;
    void *args[] = {&l, &s};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(k_match_sw), dim3(grid), dim3(ST), args, 0, st);
}

}  // namespace pccl
