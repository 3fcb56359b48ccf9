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
//     owned by one wavefront (lane i <-> in-link i), which keeps d's
//     in-links, d's needs row and the arrivals into d; clashes are resolved
//     inside the wavefront, with no workgroup barrier.
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
// its source receives a needed chunk), so its next scan starts there, and
// an upper bound on its number of candidates (counted in the setup, raised
// by such arrivals, lowered by its own commits), so a freed link whose bound
// is zero, or whose candidates are all listed arrivals, is not scanned.
// Each lane first probes the next few words of its own link's two rows; only
// the scans that run past the probe are continued by the whole wavefront.
//
// A device with more than 64 in-links or more than 512 arrival pairs (a
// switch with many ports) is split over the wavefronts of a workgroup of its
// own, one part of its in-links each.  The parts share the device's needs
// row and send-log segment, run the same event times and pick rounds, and
// settle clashes between parts through winner tables in LDS, with workgroup
// barriers per event and per round (a separate build of the kernel, so that
// the other devices carry none of it).
//
// With a switch model (Sec. 4.7) whose only binding rule is the
// no-multicast one, this kernel is queued next to the switch-group kernel
// and runs only when the device found that the rule cannot act.
#include "pccl_internal.h"

namespace pccl {
namespace {

constexpr uint32_t NT = MATCH_THREADS;
constexpr uint32_t NWAVES = NT / 64;
constexpr uint32_t MAXIN = MAX_IN_LINKS;  // one lane per in-link
constexpr uint32_t PAIRS = MAX_PAIRS;
constexpr uint32_t M_IDLE = 0, M_FULL = 1, M_ARR = 2, M_ARR_WON = 3;
constexpr uint32_t K_NONE = 0, K_BUSY = 1, K_IDLE = 2;
constexpr uint32_t SPIN_LIMIT = 1u << 24;
constexpr uint32_t PROBE_WORDS = 8;  // words per row one lane probes per step
constexpr uint32_t SEG_STEPS = 4;    // lane-group probe steps before the whole wave helps
constexpr uint32_t LA_WORDS = 8;     // words per row of one look-ahead step
constexpr uint32_t PAIRS_PER_LANE = PAIRS / 64;
constexpr uint32_t SWEEPS = 4;       // 128-word sweeps of a whole-wave scan in flight together
constexpr uint32_t SWEEPS_LDS = 2;   // the same with the needs row in LDS (only holds words are loaded), first round trip
constexpr uint32_t SWEEPS_LDS_MORE = 8;  // with the needs row in LDS, every later round trip of a scan
constexpr uint32_t FEW_SCANS = 1;    // up to this many full scans go straight to whole-wave scans
constexpr uint32_t CLASH_SLOTS = 1024;  // hash slots of the clash detection table (10 bits)
constexpr uint32_t FEW_PICKS = 8;       // up to this many picking links compare picks lane to lane
constexpr uint32_t POLL_BATCH = 4;      // exchange slots one polling lane loads per batch (256 workgroups)

static_assert(MAXIN == 64, "one lane per in-link");

// Needs rows of the workgroup's destinations, one per wave, when they fit in
// LDS (dynamic shared memory, sized at launch).  A destination's needs row
// is read and written only by the wave that owns it, so the copy is exact;
// the row in device memory is not updated while the kernel runs.
extern __shared__ __attribute__((aligned(16))) uint64_t needs_lds[];

// Per-wavefront scratch (one destination at a time).  When every wave owns
// one destination for the whole run, the per-link part persists across
// windows (no reload).
struct alignas(16) WaveShared {
    uint32_t src[MAXIN], srcoff[MAXIN], tim[MAXIN];
    uint32_t cur[MAXIN], pick[MAXIN], mode[MAXIN], kind[MAXIN];
    uint32_t cum[MAXIN + 1];
    // upper bound on each link's candidates (chunks its source holds that
    // the destination needs): arrivals at the source that the destination
    // needs add one, the link's own commits subtract one, a pick round that
    // finds no candidate sets it to 0 (commits by other links are not
    // subtracted, so it only over-counts)
    uint32_t known[MAXIN];
    // per pick round: the lowest listed candidate of each link (arrivals
    // not yet in the source's row) and how many listed candidates it has
    uint32_t xpick[MAXIN], xcnt[MAXIN];
    // split destinations: per part, its winners of the round (table order)
    // that also win across parts; this part's first send-log slot of the round
    uint64_t fin[NWAVES];
    unsigned long long logq;
    uint32_t arr_end[PAIRS], arr_c[PAIRS];
    uint32_t unf_c[PAIRS];
    uint8_t arr_j[PAIRS], unf_j[PAIRS], arr_need[PAIRS], unf_need[PAIRS];
    uint32_t seg_j[MAXIN], seg_p[MAXIN], seg_pos[MAXIN];  // probe groups: link, result, continuation word
    // clash detection: lane that last wrote a hashed pick, and slots written
    // twice.  For a part of a split destination, clash_lane also holds the
    // part's winners of a pick round once its own clashes are resolved
    alignas(16) uint8_t clash_lane[CLASH_SLOTS];
    uint8_t clash_hit[CLASH_SLOTS];
    // round (low 16 bits) in which a chunk of each hash slot was last delivered
    uint16_t dlv_round[CLASH_SLOTS];
};



// Winners of one pick round of a part of a split destination (chunk, link
// time, link id), read by the other parts of the destination.
struct WinTable {
    uint32_t chunk[MAXIN], tim[MAXIN], lid[MAXIN];
};
static_assert(sizeof(WinTable) <= CLASH_SLOTS, "the winners' table lives in the clash table's space");
__device__ __forceinline__ WinTable &win_table(WaveShared &w) { return *reinterpret_cast<WinTable *>(w.clash_lane); }

// What the parts of a split destination exchange (one per workgroup: a split
// destination has a workgroup to itself, one part per wave).
struct GroupShared {
    unsigned long long log_next;  // next free slot of the destination's send-log segment
    uint32_t tmin[NWAVES];        // per part: its next event time
    uint32_t wcnt[NWAVES];        // per part: its winners of the round (in its table)
    uint32_t flag[NWAVES];        // per part: bit 0 a link picked, bit 1 a link lost a clash inside the part
};

__device__ inline void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wave-wide reductions with DPP row operations (no LDS round trip): two quad
// permutations, row shifts by 4 and 8, then the row broadcasts of lanes 15
// and 31 leave the result over all 64 lanes in lane 63, which is read back as
// a uniform value.  Lanes without a DPP source contribute the identity.
template <class Op>
__device__ inline uint32_t dpp_reduce(uint32_t v, uint32_t id, Op op)
{
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0xb1, 0xf, 0xf, false));   // quad_perm 1,0,3,2
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x4e, 0xf, 0xf, false));   // quad_perm 2,3,0,1
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x114, 0xf, 0xf, false));  // row_shr 4
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x118, 0xf, 0xf, false));  // row_shr 8
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast 15
    v = op(v, (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast 31
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

template <class Op>
__device__ inline uint64_t dpp_reduce64(uint64_t v, uint64_t id, Op op)
{
#define PCCL_DPP64(ctrl, rmask)                                                                          \
    {                                                                                                    \
        const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)id, (int)(uint32_t)v,  \
                                                                  ctrl, rmask, 0xf, false);              \
        const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(id >> 32),            \
                                                                  (int)(uint32_t)(v >> 32), ctrl, rmask, \
                                                                  0xf, false);                           \
        v = op(v, ((uint64_t)hi << 32) | lo);                                                            \
    }
    PCCL_DPP64(0xb1, 0xf)
    PCCL_DPP64(0x4e, 0xf)
    PCCL_DPP64(0x114, 0xf)
    PCCL_DPP64(0x118, 0xf)
    PCCL_DPP64(0x142, 0xa)
    PCCL_DPP64(0x143, 0xc)
#undef PCCL_DPP64
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

struct OpMin { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return min(a, b); } };
struct OpMax { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return max(a, b); } };
struct OpAdd { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; } };
struct OpMin64 { __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a < b ? a : b; } };
struct OpAdd64 { __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; } };

__device__ inline uint32_t wave_min(uint32_t v) { return dpp_reduce(v, NONE32, OpMin()); }
__device__ inline uint32_t wave_max(uint32_t v) { return dpp_reduce(v, 0u, OpMax()); }
__device__ inline unsigned long long wave_sum64(unsigned long long v) { return dpp_reduce64(v, 0ull, OpAdd64()); }
__device__ inline uint64_t wave_min64(uint64_t v) { return dpp_reduce64(v, NONE64, OpMin64()); }

// The value of `v` in lane `lane`, which must be the same in every lane.
__device__ inline uint32_t readlane32(uint32_t v, uint32_t lane)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)lane);
}

__device__ inline uint64_t readlane64(uint64_t v, uint32_t lane)
{
    return ((uint64_t)readlane32((uint32_t)(v >> 32), lane) << 32) | readlane32((uint32_t)v, lane);
}

__device__ inline uint32_t lane_prefix(uint64_t mask, uint32_t lane)
{
    return (uint32_t)__popcll(mask & ((1ull << lane) - 1ull));
}


// 128-bit pieces of the two rows, handled as four 32-bit dwords (x holds the
// lowest bits): wave64 VALU work is issued at one instruction per four
// cycles, so the scans avoid 64-bit compares, selects and bit counts.
__device__ inline uint4 and4(uint4 a, uint4 b) { return make_uint4(a.x & b.x, a.y & b.y, a.z & b.z, a.w & b.w); }

// Keeps the bits of the 128-bit piece starting at bit `base` that lie at or
// above bit `from`.
__device__ inline uint4 keep_from(uint4 a, uint32_t base, uint32_t from)
{
    const uint32_t sh = from > base ? from - base : 0u;
    const uint32_t q = sh >> 5, t = ~0u << (sh & 31u);
    a.x &= q > 0u ? 0u : t;
    a.y &= q > 1u ? 0u : (q == 1u ? t : ~0u);
    a.z &= q > 2u ? 0u : (q == 2u ? t : ~0u);
    a.w &= q > 3u ? 0u : (q == 3u ? t : ~0u);
    return a;
}

// Offset of the lowest set bit of a 128-bit piece, NONE32 if it is zero.
__device__ inline uint32_t first4(uint4 a)
{
    uint32_t r = a.w ? 96u + (uint32_t)__builtin_ctz(a.w) : NONE32;
    r = a.z ? 64u + (uint32_t)__builtin_ctz(a.z) : r;
    r = a.y ? 32u + (uint32_t)__builtin_ctz(a.y) : r;
    r = a.x ? (uint32_t)__builtin_ctz(a.x) : r;
    return r;
}

__device__ inline bool any4(uint4 a) { return (a.x | a.y | a.z | a.w) != 0u; }

// Two words of the holds bitmap at word index w (row * Wp + word), read with
// the cache policy of an agent-scope atomic load (sc1): coherent with the
// folds other workgroups make, so the kernel that reads holds rows only this
// way needs no cache invalidation after each window exchange.  The buffer
// descriptor spans the bitmap (`bytes`, below 2 GiB); a read past its end
// returns zeros.
constexpr int BUF_RSRC_WORD3 = 0x00020000;  // gfx9 buffer descriptor: 32-bit data format, raw access
constexpr int CPOL_SC1 = 16;                // cache policy bit sc1
__device__ __forceinline__ uint4 holds_load4(const uint64_t *holds, uint32_t bytes, uint32_t w)
{
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint64_t *>(holds), (short)0, (int)bytes, BUF_RSRC_WORD3);
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)(w * 8u), 0, CPOL_SC1));
}

// Bitset intersect + select for one link, by a whole wave: the first set bit
// at position >= cur of holds[src] & needs[dst], in priority order.  Each
// lane loads 16 bytes of each row per sweep (SW sweeps in flight, 1 KiB per
// row per sweep and wave), a ballot finds the first lane with a non-zero
// AND, and a count-trailing-zeros gives the chunk.  `words` counts the words
// per row the scan needed (through the word holding the pick, or to the row
// end).
//
// With the needs row in LDS (MIRROR) only the holds words are loaded: the
// first round trip takes SWEEPS_LDS sweeps (most scans end there), a scan
// that goes on SWEEPS_LDS_MORE per round trip.
template <bool MIRROR, uint32_t SW>
__device__ __forceinline__ bool wave_sweeps(const uint64_t *__restrict__ holds, uint32_t hbytes,
                                            const uint64_t *__restrict__ h, const uint64_t *__restrict__ nd,
                                            uint32_t cur, uint32_t w0, uint32_t wp, uint32_t wb, uint64_t &words,
                                            uint32_t &pick)
{
    const uint32_t lane = threadIdx.x & 63;
    uint4 a[SW];
    if constexpr (MIRROR) {
        // every load is issued before any is used (a load past the row end
        // reads its last piece and is masked out)
        uint4 hv[SW];
        const uint32_t hrow = (uint32_t)(h - holds);
#pragma unroll
        for (uint32_t u = 0; u < SW; u++) {
            const uint32_t idx = wb + 128 * u + 2 * lane;
            hv[u] = holds_load4(holds, hbytes, hrow + min(idx, wp - 2u));
        }
#pragma unroll
        for (uint32_t u = 0; u < SW; u++) {
            const uint32_t idx = wb + 128 * u + 2 * lane;
            a[u] = idx < wp ? and4(hv[u], *reinterpret_cast<const uint4 *>(nd + idx)) : make_uint4(0, 0, 0, 0);
        }
    } else {
#pragma unroll
        for (uint32_t u = 0; u < SW; u++) {
            const uint32_t idx = wb + 128 * u + 2 * lane;
            a[u] = make_uint4(0, 0, 0, 0);
            if (idx < wp)
                a[u] = and4(*reinterpret_cast<const uint4 *>(h + idx), *reinterpret_cast<const uint4 *>(nd + idx));
        }
    }
    // only a piece of the scan's first sweep can hold bits below the cursor
    // (the scan starts at the even word below it)
    a[0] = keep_from(a[0], (wb + 2 * lane) * 64, cur);
#pragma unroll
    for (uint32_t u = 0; u < SW; u++) {
        const uint64_t m = __ballot(any4(a[u]));
        if (m) {
            const uint32_t fl = (uint32_t)__builtin_ffsll((long long)m) - 1u;
            const uint32_t r = readlane32(first4(a[u]), fl);
            const uint32_t idx = wb + 128 * u + 2 * fl;
            words += (uint64_t)(idx + (r >> 6) + 1 - w0);
            pick = idx * 64 + r;
            return true;
        }
    }
    return false;
}

template <bool MIRROR>
__device__ __forceinline__ uint32_t wave_first_candidate(const uint64_t *__restrict__ holds, uint32_t hbytes,
                                                         const uint64_t *__restrict__ h, const uint64_t *__restrict__ nd,
                                                         uint32_t cur, uint64_t Ws, uint64_t &words)
{
    constexpr uint32_t SW1 = MIRROR ? SWEEPS_LDS : SWEEPS, SW2 = MIRROR ? SWEEPS_LDS_MORE : SWEEPS;
    const uint32_t w0 = cur >> 6, wp = (uint32_t)Ws;
    if (w0 >= wp) return NONE32;
    uint32_t pick = NONE32;
    uint32_t wb = w0 & ~1u;
    if (wave_sweeps<MIRROR, SW1>(holds, hbytes, h, nd, cur, w0, wp, wb, words, pick)) return pick;
    // (past the first round trip no piece lies below the cursor: keep_from
    // passes every bit of a piece that starts above it)
    for (wb += 128 * SW1; wb < wp; wb += 128 * SW2)
        if (wave_sweeps<MIRROR, SW2>(holds, hbytes, h, nd, cur, w0, wp, wb, words, pick)) return pick;
    words += Ws - w0;
    return NONE32;
}

// Grid-wide exchange at the end of window `gen`, which is also the grid
// barrier: every workgroup publishes its results in one 64-bit slot of its
// own cache line (so the pollers' loads spread over the memory channels):
// gen+1 (12 bits) | error flag | transfers committed (19 bits) | earliest
// transfer end (32 bits).  The last wave of every workgroup then polls all slots,
// one per lane, until each carries the tag, and reduces them itself.  Slots
// alternate with the window parity: a workgroup can run at most one window
// ahead of the slowest poller, so it never overwrites a slot that is still
// being read.  No atomic read-modify-write and no second round trip to
// release the waiters.
// Memory ordering: the writes of a window that other workgroups read (the
// snapshot entries and the holds folds) are agent-scope atomics, coherent
// without an L2 write-back; every wave waits for their completion before the
// workgroup barrier, so they are performed before the slots are written.
// After the wait, the kernel that keeps needs rows in device memory takes an
// agent-scope acquire fence, so that its later plain loads miss any line
// cached before the other workgroups wrote it; the kernel with needs rows in
// LDS reads holds rows and snapshot entries only with coherent loads (the
// sc1 cache policy) and skips that cache invalidation.
struct Exchange {
    uint32_t tn;              // start of the next window (earliest transfer end), NONE32 if none
    uint32_t err;             // some workgroup recorded an error
    unsigned long long sent;  // transfers committed in the window, grid-wide
    uint32_t ok;              // 0 if the wait was abandoned
};

struct BlockShared {
    WaveShared w[NWAVES];
    GroupShared g;
    uint32_t red_tmin[NWAVES], red_err[NWAVES];
    unsigned long long red_sent[NWAVES];
    Exchange ex;
};

// First half: publish this workgroup's slot.  Called by every thread after
// the workgroup barrier that follows each wave's wait for the completion of
// its writes and atomics of the window.
constexpr uint64_t XTAG_MASK = 0xFFFull << 52;
static_assert((uint64_t)MAX_DEVICES_SP * MAX_IN_LINKS < (1u << 19), "a window's transfers fit in 19 bits");

__device__ void window_publish(uint64_t *xslot, uint32_t gen, uint32_t tmin, unsigned long long sent, uint32_t err)
{
    const uint64_t tag = (uint64_t)((gen + 1u) & 0xFFFu) << 52;
    uint64_t *slot = xslot + (uint64_t)((gen + 1u) & 1u) * MAX_MATCH_GRID * XSLOT_WORDS;
    if (threadIdx.x == 0)
        __hip_atomic_store(&slot[(uint64_t)blockIdx.x * XSLOT_WORDS],
                           tag | ((uint64_t)(err ? 1u : 0u) << 51) | ((uint64_t)(sent & 0x7FFFFu) << 32) | tmin,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Second half: wait for every workgroup's slots and reduce them.
template <bool COHERENT>
__device__ bool window_wait(Control *ctl, uint64_t *xslot, BlockShared &sh, uint32_t gen, Exchange &ex)
{
    const uint32_t nb = gridDim.x, lane = threadIdx.x & 63;
    const uint64_t tag = (uint64_t)((gen + 1u) & 0xFFFu) << 52;
    uint64_t *slot = xslot + (uint64_t)((gen + 1u) & 1u) * MAX_MATCH_GRID * XSLOT_WORDS;
    // the last wave polls: in a workgroup that holds one heavy destination on
    // wave 0 and idle waves after it, the destination's wave is then free to
    // finish its look-ahead during the wait
    if ((threadIdx.x >> 6) == (blockDim.x >> 6) - 1u) {
        uint32_t spins = 0, ok = 1;
        uint32_t tn = NONE32, e = 0;
        unsigned long long s = 0;
        while (true) {
            bool all = true;
            tn = NONE32;
            e = 0;
            s = 0;
            // every load of one spin is issued before any result is used, so
            // a spin costs one memory round trip, not one per slot.  The loads
            // are unconditional (lanes past the last workgroup reread its slot
            // and are ignored): a load under a branch would make the compiler
            // wait for it where the branches join.
            const uint32_t ab = __hip_atomic_load(&ctl->abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (uint32_t b0 = 0; b0 < nb; b0 += 64 * POLL_BATCH) {
                uint64_t a[POLL_BATCH];
#pragma unroll
                for (uint32_t u = 0; u < POLL_BATCH; u++)
                    a[u] = __hip_atomic_load(&slot[(uint64_t)min(b0 + 64 * u + lane, nb - 1u) * XSLOT_WORDS],
                                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                for (uint32_t u = 0; u < POLL_BATCH; u++) {
                    if (b0 + 64 * u + lane >= nb) continue;
                    if ((a[u] & XTAG_MASK) != tag) all = false;
                    tn = min(tn, (uint32_t)a[u]);
                    e |= (uint32_t)(a[u] >> 51) & 1u;
                    s += (a[u] >> 32) & 0x7FFFFull;
                }
            }
            if (__ballot(!all) == 0) break;
            if (ab) {
                ok = 0;
                break;
            }
            if (++spins > SPIN_LIMIT) {
                if (lane == 0) atomicExch(&ctl->abort, 1u);
                ok = 0;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        // acquire: this compute unit's caches drop lines other workgroups
        // wrote; a kernel that reads those lines only with coherent loads
        // orders its later loads after the wait without that invalidation
        if constexpr (COHERENT) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        else __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        tn = wave_min(tn);
        e = __ballot(e != 0) ? 1u : 0u;
        s = wave_sum64(s);
        if (lane == 0) {
            sh.ex.tn = tn;
            sh.ex.err = e;
            sh.ex.sent = s;
            sh.ex.ok = ok;
        }
    }
    __syncthreads();
    ex = sh.ex;
    return ex.ok != 0;
}

// Per-wavefront accumulators, kept identical on every lane.
struct Acc {
    uint32_t tmin;     // earliest end among transfers in flight on this wave's links
    uint32_t cstar;    // latest transfer end committed by this wave
    uint32_t err;      // this wave recorded an error
    unsigned long long sent, rounds, clashes, words;
    // per-lane parts, reduced once at the end of the kernel
    unsigned long long lane_words;  // word positions this lane's scans passed
    uint32_t lane_cstar;            // latest end of a transfer this lane committed
};

// One wavefront's destination: uniform values and this lane's in-link.
struct Dest {
    uint32_t d, base, n, pairs;
    uint32_t part, nparts;      // split destination: this wave's part and the number of parts (else 0, 0)
    uint32_t src, tim, lid;     // this lane's in-link (lane < n): source, time, link id
    uint32_t busy, infl, idle;  // its state
    uint32_t ready;             // the cursor points at a candidate found ahead of time
    uint32_t ready_c;           // that candidate while it is valid (NONE32 when not kept)
    uint32_t fold;              // chunk delivered into d in the previous window, still to fold
    uint32_t n_arr_prev;        // length of the previous window's arrival list (kept in LDS)
    uint32_t n_unf_prev;        // length of the previous window's list of unfolded arrivals
    unsigned long long log;     // next send-log slot of d
    // arrival pairs p = 64 u + lane: slot of the source's in-link, and the
    // in-link of d it feeds (slot << 8 | j; NONE32 past the last pair)
    uint32_t pair[PAIRS_PER_LANE];
};

// `wp`: the wave's part of a split destination (parts << 24 | part << 16 |
// first in-link << 8 | in-links), 0 for a whole destination.
__device__ void load_dest(const Layout &ly, WaveShared &ws, uint32_t d, uint32_t wp, Dest &ds)
{
    const uint32_t lane = threadIdx.x & 63;
    ds.d = d;
    const uint32_t b0 = ly.in_off[d], nall = ly.in_off[d + 1] - b0;
    const uint32_t first = wp ? (wp >> 8) & 0xFFu : 0u;
    ds.nparts = wp >> 24;
    ds.part = (wp >> 16) & 0xFFu;
    ds.base = b0 + first;
    ds.n = wp ? (wp & 0xFFu) : nall;
    // arrival pairs of this part's in-links (the prefix is per destination)
    const uint32_t cum0 = first < nall ? ly.slot_cum[ds.base] : ly.dest_pairs[d];
    const uint32_t cum1 = first + ds.n < nall ? ly.slot_cum[ds.base + ds.n] : ly.dest_pairs[d];
    ds.pairs = cum1 - cum0;
    ds.log = ly.dest_log[d];
    ds.src = 0;
    ds.tim = 0;
    ds.lid = 0;
    ds.busy = 0;
    ds.infl = NONE32;
    ds.idle = 0;
    ds.ready = 0;
    ds.ready_c = NONE32;
    ds.fold = NONE32;
    ds.n_arr_prev = 0;
    ds.n_unf_prev = 0;
    if (lane < ds.n) {
        const uint32_t sl = ds.base + lane;
        ds.src = ly.slot_src[sl];
        ds.tim = ly.slot_time[sl];
        ds.busy = ly.busy[sl];
        ds.infl = ly.infl[sl];
        ds.idle = ly.lflags[sl] & 1u;
        ds.ready = (ly.lflags[sl] >> 1) & 1u;
        ws.src[lane] = ds.src;
        ws.srcoff[lane] = ly.in_off[ds.src];
        ws.tim[lane] = ds.tim;
        ds.lid = ly.slot_link[sl];
        ws.cur[lane] = ly.cur[sl];
        ws.cum[lane] = ly.slot_cum[sl] - cum0;
        ws.known[lane] = ly.lcnt[sl];
    }
    if (lane == 0) ws.cum[ds.n] = ds.pairs;
    wave_sync();
#pragma unroll
    for (uint32_t u = 0; u < PAIRS_PER_LANE; u++) {
        const uint32_t p = 64 * u + lane;
        ds.pair[u] = NONE32;
        if (p < ds.pairs) {
            uint32_t lo = 0, hi = ds.n;
            while (hi - lo > 1) {
                const uint32_t mid = (lo + hi) >> 1;
                if (ws.cum[mid] <= p) lo = mid;
                else hi = mid;
            }
            ds.pair[u] = ((ws.srcoff[lo] + (p - ws.cum[lo])) << 8) | lo;
        }
    }
}

__device__ void store_dest(const Layout &ly, WaveShared &ws, const Dest &ds)
{
    const uint32_t lane = threadIdx.x & 63;
    if (lane < ds.n) {
        const uint32_t sl = ds.base + lane;
        ly.busy[sl] = ds.busy;
        ly.infl[sl] = ds.infl;
        ly.cur[sl] = ws.cur[lane];
        ly.lflags[sl] = ds.idle | (ds.ready << 1);
        ly.lcnt[sl] = ws.known[lane];
    }
    if (lane == 0) ly.dest_log[ds.d] = ds.log;
    wave_sync();
}

// Look-ahead for busy links: one probe step of LA_WORDS words from the
// cursor, combined with the window's listed arrivals, so that the scan at
// completion starts at the next candidate.  The cursor stays a lower bound:
// candidates only appear through arrivals, which lower it when they come.
// The loads are issued at the end of a window and, when the wave keeps its
// destination, consumed at the start of the next one, so their round trip
// overlaps the window exchange.  The lists of the issuing window stay in
// LDS until then.
struct LookAhead {
    uint4 hv[LA_WORDS / 2], nv[LA_WORDS / 2];  // the two rows' words from the even word below the cursor
    uint32_t cur;           // cursor the words were loaded from, NONE32 if none
    uint32_t n_arr, n_unf;  // list lengths of the issuing window
    unsigned long long words;  // word positions this lane's look-aheads passed (summed at the end)
};

template <bool MIRROR>
__device__ __forceinline__ void look_ahead_issue(const Layout &ly, uint32_t hbytes, uint64_t Wp, uint64_t Ws,
                                                 const WaveShared &ws,
                                                 const Dest &ds, const uint64_t *nd, bool mine, uint32_t n_arr,
                                                 uint32_t n_unf, LookAhead &la)
{
    const uint32_t lane = threadIdx.x & 63;
    la.cur = NONE32;
    la.n_arr = n_arr;
    la.n_unf = n_unf;
    // (a link with no candidate left has nothing to look for)
    if (!(mine && ds.infl != NONE32 && !ds.ready && ws.known[threadIdx.x & 63] != 0)) return;
    const uint32_t cur = ws.cur[lane];
    if ((cur >> 6) >= Ws) return;
    la.cur = cur;
    const uint64_t pos = (cur >> 6) & ~1u;
    const uint64_t *h = ly.holds + (uint64_t)ds.src * Wp;
#pragma unroll
    for (uint32_t u = 0; u < LA_WORDS / 2; u++) {
        const uint64_t idx = pos + 2 * u;
        if (idx < Ws) {
            if constexpr (MIRROR) la.hv[u] = holds_load4(ly.holds, hbytes, (uint32_t)(ds.src * Wp + idx));
            else la.hv[u] = *reinterpret_cast<const uint4 *>(h + idx);
            if constexpr (!MIRROR) la.nv[u] = *reinterpret_cast<const uint4 *>(nd + idx);
        } else {
            la.hv[u] = make_uint4(0, 0, 0, 0);
            if constexpr (!MIRROR) la.nv[u] = make_uint4(0, 0, 0, 0);
        }
    }
}

template <bool MIRROR>
__device__ __forceinline__ void look_ahead_finish(uint64_t Ws, WaveShared &ws, Dest &ds, const uint64_t *nd, bool mine,
                                                  LookAhead &la)
{
    const uint32_t lane = threadIdx.x & 63;
    const bool pf = mine && la.cur != NONE32;
    if (!__ballot(pf)) return;
    uint32_t p = NONE32;
    const uint64_t pos = (la.cur >> 6) & ~1u;
    if (pf) {
        // the words were loaded from bit (cur & ~127): only the first piece
        // holds bits below the cursor
        const uint32_t base = la.cur & ~127u;
        if constexpr (MIRROR) {
            // the needs words come from the destination's row in LDS (no
            // commit can have changed it since the holds words were loaded)
#pragma unroll
            for (uint32_t u = 0; u < LA_WORDS / 2; u++)
                la.nv[u] = pos + 2 * u < Ws ? *reinterpret_cast<const uint4 *>(nd + pos + 2 * u) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = (int)(LA_WORDS / 2) - 1; u >= 0; u--) {
            uint4 a = and4(la.hv[u], la.nv[u]);
            if (u == 0) a = keep_from(a, base, la.cur);
            const uint32_t r = first4(a);
            if (r != NONE32) p = base + 128u * (uint32_t)u + r;
        }
    }
    if (mine) ws.pick[lane] = pf ? p : NONE32;
    ws.kind[lane] = pf ? 1u : 0u;
    wave_sync();
    for (uint32_t q = lane; q < la.n_arr; q += 64) {
        const uint32_t j = ws.arr_j[q], c = ws.arr_c[q];
        if (ws.arr_need[q] && ws.kind[j] && c >= ws.cur[j]) atomicMin(&ws.pick[j], c);
    }
    for (uint32_t q = lane; q < la.n_unf; q += 64) {
        const uint32_t j = ws.unf_j[q], c = ws.unf_c[q];
        if (ws.unf_need[q] && ws.kind[j] && c >= ws.cur[j]) atomicMin(&ws.pick[j], c);
    }
    wave_sync();
    if (pf) {
        // only the probed words are known empty: a listed arrival beyond
        // them does not let the cursor skip unprobed words
        const uint64_t end_w = pos + LA_WORDS;
        const uint32_t probed = end_w >= Ws ? (uint32_t)(Ws * 64) : (uint32_t)(end_w * 64);
        const uint32_t pk = ws.pick[lane];
        const uint64_t w0 = la.cur >> 6;
        if (pk < probed) {
            ws.cur[lane] = pk;
            ds.ready = 1;
            ds.ready_c = pk;
            la.words += (pk >> 6) + 1 - w0;
        } else {
            ws.cur[lane] = probed;
            la.words += min(end_w, Ws) - w0;
        }
    }
    la.cur = NONE32;
    wave_sync();
}

// A snapshot entry another workgroup wrote: with COHERENT, an agent-scope
// atomic load (the kernel that reads this way invalidates no caches after the
// window exchange), else a plain load after the exchange's acquire fence.
template <bool COHERENT>
__device__ __forceinline__ uint64_t snap_load(const uint64_t *p)
{
    if constexpr (COHERENT) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else return *p;
}

// All events of window [t0, t1) for one destination, by one wavefront.
// `grp`: the WaveShared of part 0 of a split destination (its parts are
// consecutive waves), `gs` what the parts exchange; unused otherwise.  The
// parts of a split destination run the same event times and pick rounds in
// step: a workgroup barrier gives every part the next event time, another
// follows the publication of each part's winners of a round (every part then
// resolves the clashes between parts the same way: fastest link, then lowest
// id), a third the commits of the round (so the next round's picks see the
// shared needs row as all parts left it).
template <bool MIRROR, bool SPLIT>
__device__ void process_window(const Layout &ly, const Sizes &sz, WaveShared &ws, Dest &ds, uint32_t k,
                               uint32_t t0, uint64_t t1, bool resident, Acc &acc, LookAhead &la, WaveShared *grp,
                               GroupShared &gs)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t n = ds.n, d = ds.d;
    // (only the kernel variants built for split destinations take parts;
    // the host deals parts to no other)
    const bool split = SPLIT && ds.nparts > 1;
    if (n == 0 && !split) return;
    // Wp: row stride; Ws: where scans end (bits past the last chunk are zero
    // in both rows, so no candidate lies beyond the row's own words)
    const uint64_t Wp = sz.Wp, Ws = (sz.W + 1) & ~1ull, L = sz.L;
    const uint32_t END = (uint32_t)(Ws * 64);
    uint64_t *nd;
    if constexpr (MIRROR) nd = needs_lds + (uint64_t)((threadIdx.x >> 6) - ds.part) * Wp;  // part 0's row
    else nd = ly.needs + (uint64_t)d * Wp;
    uint64_t *hd = ly.holds + (uint64_t)d * Wp;
    const uint64_t *snap1 = ly.snap + (uint64_t)((k + 2) % 3) * L;  // in flight at the end of window k-1
    const uint64_t *snap2 = ly.snap + (uint64_t)((k + 1) % 3) * L;  // in flight at the end of window k-2 (unless carried)
    uint64_t *snap0 = ly.snap + (uint64_t)(k % 3) * L;              // written for window k+1
    const bool mine = lane < n;
    const uint32_t sl = ds.base + lane;
    // fold the arrivals of window k-1 into d's holds row (a resident wave
    // remembers them; otherwise they are the snapshot entries that ended)
    if (mine) {
        ws.mode[lane] = M_IDLE;
        uint32_t r = NONE32;
        if (resident) {
            r = ds.fold;
        } else if (k >= 2) {
            const uint64_t e = snap_load<MIRROR>(&snap2[sl]);
            if (e != NONE64 && (uint32_t)e < t0) r = (uint32_t)(e >> 32);
        }
        if (r != NONE32)
            __hip_atomic_fetch_or(&hd[r >> 6], 1ull << (r & 63), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ds.fold = NONE32;
    }

    // this window's snapshot entry, as far as known now: a transfer that
    // outlasts the window stays in flight; any other link ends the window
    // free unless it commits in it, and then the commit writes the entry
    if (mine)
        __hip_atomic_store(&snap0[sl],
                           ds.infl != NONE32 && (uint64_t)ds.busy >= t1 ? (((uint64_t)ds.infl << 32) | ds.busy) : NONE64,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    // the snapshot entries of the arrival pairs (below) are loaded next, so
    // that their round trip overlaps the look-ahead; the fold and the entry
    // above go out first, so waiting for these loads waits for them too
    const bool carry = resident && k >= 2;
    uint64_t e1[PAIRS_PER_LANE], e2[PAIRS_PER_LANE];
#pragma unroll
    for (uint32_t u = 0; u < PAIRS_PER_LANE; u++) {
        e1[u] = NONE64;
        e2[u] = NONE64;
        const uint32_t pr = ds.pair[u];
        if (k >= 1 && pr != NONE32) {
            e1[u] = snap_load<MIRROR>(&snap1[pr >> 8]);
            if (k >= 2 && !carry) e2[u] = snap_load<MIRROR>(&snap2[pr >> 8]);
        }
    }
    // the look-ahead issued at the end of the last window
    if (resident) look_ahead_finish<MIRROR>(Ws, ws, ds, nd, mine, la);

    // arrivals at the sources of d's in-links that d needs: this window's
    // (snapshot k-1, ends in [t0, t1)) and last window's (snapshot k-2,
    // ends before t0; possibly not folded into the source's row yet).
    // Every snapshot k-2 entry that ends before t0 ended in the last window,
    // so when the wave keeps its destination, last window's list, with the
    // flags of the chunks delivered since cleared, is exactly this window's
    // second list: it is carried over in LDS instead of reloaded.
    uint32_t n_arr = 0, n_unf = 0;
    if (carry) {
        for (uint32_t q0 = 0; q0 < ds.n_arr_prev; q0 += 64) {
            const uint32_t q = q0 + lane;
            const bool keep = q < ds.n_arr_prev && ws.arr_need[q];
            uint32_t c = 0;
            uint8_t j = 0;
            if (keep) {
                c = ws.arr_c[q];
                j = ws.arr_j[q];
            }
            const uint64_t m = __ballot(keep);
            if (keep) {
                const uint32_t u = n_unf + lane_prefix(m, lane);
                ws.unf_c[u] = c;
                ws.unf_j[u] = j;
                ws.unf_need[u] = 1;
            }
            n_unf += (uint32_t)__popcll(m);
        }
        wave_sync();
    }
    if (k >= 1) {
        {
            // the needs words of all entries are read before any is used (an
            // empty entry reads chunk 0's word), so their latencies overlap
            bool a_ok[PAIRS_PER_LANE], u_ok[PAIRS_PER_LANE];
            uint64_t nw1[PAIRS_PER_LANE], nw2[PAIRS_PER_LANE];
#pragma unroll
            for (uint32_t u = 0; u < PAIRS_PER_LANE; u++) {
                nw1[u] = nd[(e1[u] != NONE64 ? (uint32_t)(e1[u] >> 32) : 0u) >> 6];
                if (!carry) nw2[u] = nd[(e2[u] != NONE64 ? (uint32_t)(e2[u] >> 32) : 0u) >> 6];
            }
#pragma unroll
            for (uint32_t u = 0; u < PAIRS_PER_LANE; u++) {
                const uint32_t c1 = (uint32_t)(e1[u] >> 32), c2 = (uint32_t)(e2[u] >> 32);
                a_ok[u] = e1[u] != NONE64 && (uint64_t)(uint32_t)e1[u] < t1 && ((nw1[u] >> (c1 & 63)) & 1ull);
                u_ok[u] = !carry && e2[u] != NONE64 && (uint32_t)e2[u] < t0 && ((nw2[u] >> (c2 & 63)) & 1ull);
            }
#pragma unroll
            for (uint32_t u = 0; u < PAIRS_PER_LANE; u++) {
                if (64 * u >= ds.pairs) break;
                const uint64_t ma = __ballot(a_ok[u]), mu = __ballot(u_ok[u]);
                const uint8_t j = (uint8_t)(ds.pair[u] & 0xFFu);
                if (a_ok[u]) {
                    const uint32_t q = n_arr + lane_prefix(ma, lane);
                    ws.arr_end[q] = (uint32_t)e1[u];
                    ws.arr_c[q] = (uint32_t)(e1[u] >> 32);
                    ws.arr_j[q] = j;
                    ws.arr_need[q] = 1;
                }
                if (u_ok[u]) {
                    const uint32_t q = n_unf + lane_prefix(mu, lane);
                    ws.unf_c[q] = (uint32_t)(e2[u] >> 32);
                    ws.unf_j[q] = j;
                    ws.unf_need[q] = 1;
                }
                n_arr += (uint32_t)__popcll(ma);
                n_unf += (uint32_t)__popcll(mu);
            }
        }
    }
    wave_sync();

    // event times of this destination inside the window, in order
    int64_t t_prev = (int64_t)t0 - 1;
    uint32_t n_send = 0;
    while (true) {
        uint32_t m = NONE32;
        if (k == 0) {
            if (t_prev < 0) m = 0;
        } else {
            if (mine && ds.infl != NONE32 && (int64_t)ds.busy > t_prev && (uint64_t)ds.busy < t1) m = ds.busy;
            for (uint32_t q = lane; q < n_arr; q += 64)
                if (ws.arr_need[q] && (int64_t)ws.arr_end[q] > t_prev) m = min(m, ws.arr_end[q]);
        }
        uint32_t t = wave_min(m);
        if (split) {
            // the destination's next event: the earliest over its parts
            if (lane == 0) gs.tmin[ds.part] = t;
            __syncthreads();
            for (uint32_t q = 0; q < ds.nparts; q++) t = min(t, gs.tmin[q]);
        }
        if (t == NONE32) break;

        // links whose transfer ends now are free and need a full scan
        uint32_t md = M_IDLE;
        if (mine) {
            if (k == 0) {
                md = M_FULL;
            } else if (ds.infl != NONE32 && ds.busy == t) {
                md = M_FULL;
                ds.fold = ds.infl;
                ds.infl = NONE32;
            }
            ws.mode[lane] = md;
            ws.kind[lane] = (md == M_FULL || ds.infl != NONE32) ? K_BUSY : (ds.idle ? K_IDLE : K_NONE);
        }
        wave_sync();
        // a needed chunk arriving at a link's source: busy or just-freed links
        // lower their cursor; an idle free link gets it as its candidate
        for (uint32_t q = lane; q < n_arr; q += 64) {
            if (ws.arr_end[q] != t || !ws.arr_need[q]) continue;
            const uint32_t j = ws.arr_j[q], c = ws.arr_c[q];
            const uint32_t kind = ws.kind[j];
            atomicAdd(&ws.known[j], 1u);
            if (kind == K_BUSY) atomicMin(&ws.cur[j], c);
            else if (kind == K_IDLE) ws.mode[j] = M_ARR;
        }
        wave_sync();
        if (mine) {
            md = ws.mode[lane];
            // a freed link whose bound says no candidate is left goes idle
            // without a scan, as a scan would have found
            if (md == M_FULL && ws.known[lane] == 0) {
                md = M_IDLE;
                ds.idle = 1;
                ws.cur[lane] = END;
                ws.mode[lane] = M_IDLE;
            }
        }

        // pick rounds at time t
        while (true) {
            // bitmap part of the full scans.  First every scanning lane
            // probes PROBE_WORDS words of its own link's two rows (most scans
            // end there: the look-ahead put the cursor on the candidate);
            // when more than FEW_SCANS links are still scanning, the wave is
            // split among them, G = 64 / next_pow2(k) lanes each, every lane
            // reading PROBE_WORDS words per step, and a min over each lane
            // group gives the link's first candidate.  Scans that are left
            // (at most FEW_SCANS, or after SEG_STEPS group steps) continue
            // with the whole wave, one link at a time.
            uint32_t p = NONE32, scanned = 0;
            bool scanning = false;
            uint64_t pos = 0, w0 = 0;
            // explicit candidates first: arrivals not yet in the source's
            // row, the lowest and the number per link
            if (mine) {
                ws.xpick[lane] = NONE32;
                ws.xcnt[lane] = 0;
            }
            wave_sync();
            for (uint32_t q = lane; q < n_arr; q += 64) {
                if (!ws.arr_need[q]) continue;
                const uint32_t j = ws.arr_j[q], c = ws.arr_c[q], mj = ws.mode[j];
                if (mj == M_FULL) {
                    if (ws.arr_end[q] <= t && c >= ws.cur[j]) {
                        atomicMin(&ws.xpick[j], c);
                        atomicAdd(&ws.xcnt[j], 1u);
                    }
                } else if (mj == M_ARR) {
                    if (ws.arr_end[q] == t) atomicMin(&ws.xpick[j], c);
                }
            }
            for (uint32_t q = lane; q < n_unf; q += 64) {
                if (!ws.unf_need[q]) continue;
                const uint32_t j = ws.unf_j[q], c = ws.unf_c[q];
                if (ws.mode[j] == M_FULL && c >= ws.cur[j]) {
                    atomicMin(&ws.xpick[j], c);
                    atomicAdd(&ws.xcnt[j], 1u);
                }
            }
            wave_sync();
            // when the link's bound does not exceed its listed candidates,
            // every candidate is listed (candidates are the union of the
            // row's and the listed ones) and the row needs no scan
            if (mine && md == M_FULL && ws.known[lane] > ws.xcnt[lane]) {
                const uint32_t cur = ws.cur[lane];
                w0 = cur >> 6;
                if (cur == ds.ready_c) {
                    // the look-ahead's candidate, still at the cursor and not
                    // delivered since: held by the source (holds only grow),
                    // still needed, and nothing lies below the cursor
                    p = cur;
                    scanned = 1;
                } else {
                    scanning = w0 < Ws;
                    pos = w0 & ~1ull;
                }
            }
            const uint64_t *h = ly.holds + (uint64_t)ds.src * Wp;
            if (__popcll(__ballot(scanning)) > FEW_SCANS && scanning) {
                uint4 hv[PROBE_WORDS / 2], nv[PROBE_WORDS / 2];
#pragma unroll
                for (uint32_t u = 0; u < PROBE_WORDS / 2; u++) {
                    const uint64_t idx = pos + 2 * u;
                    if (idx < Ws) {
                        if constexpr (MIRROR) hv[u] = holds_load4(ly.holds, sz.hbytes, (uint32_t)(ds.src * Wp + idx));
                        else hv[u] = *reinterpret_cast<const uint4 *>(h + idx);
                        nv[u] = *reinterpret_cast<const uint4 *>(nd + idx);
                    } else {
                        hv[u] = make_uint4(0, 0, 0, 0);
                        nv[u] = make_uint4(0, 0, 0, 0);
                    }
                }
                // pos = the even word below the cursor: only the first piece
                // holds bits below it
                const uint32_t cur = ws.cur[lane], base = (uint32_t)pos * 64u;
#pragma unroll
                for (int u = (int)(PROBE_WORDS / 2) - 1; u >= 0; u--) {
                    uint4 a = and4(hv[u], nv[u]);
                    if (u == 0) a = keep_from(a, base, cur);
                    const uint32_t r = first4(a);
                    if (r != NONE32) p = base + 128u * (uint32_t)u + r;
                }
                if (p != NONE32) scanned = (p >> 6) + 1u - (uint32_t)w0;
                if (p != NONE32) {
                    scanning = false;
                } else {
                    pos += PROBE_WORDS;
                    if (pos >= Ws) {
                        scanning = false;
                        scanned = (uint32_t)(Ws - w0);
                    }
                }
            }
            if (scanning) scanned = pos > w0 ? (uint32_t)(pos - w0) : 0u;  // so far; the group steps add theirs
            const uint64_t smask = __ballot(scanning);
            const uint32_t ks = (uint32_t)__popcll(smask);
            // one or two scans left: the whole-wave scan below is quicker
            if (ks > FEW_SCANS) {
                if (scanning) {
                    ws.seg_j[lane_prefix(smask, lane)] = lane;
                    ws.seg_pos[lane] = (uint32_t)pos;
                }
                wave_sync();
                const uint32_t lg = (31u - (uint32_t)__builtin_clz(ks)) + ((ks & (ks - 1u)) ? 1u : 0u);
                const uint32_t G = 64u >> lg;  // lanes per link still scanning
                const uint32_t g = lane >> (6u - lg), sub = lane & (G - 1u);
                const bool act = g < ks;
                uint32_t j = 0;
                uint64_t gw0 = 0, gpos = 0, gstart = 0;
                const uint64_t *hj = ly.holds;
                uint32_t hjrow = 0;
                if (act) {
                    j = ws.seg_j[g];
                    const uint32_t cj = ws.cur[j];
                    gw0 = cj >> 6;
                    gpos = gstart = ws.seg_pos[j];
                    hjrow = (uint32_t)(ws.src[j] * Wp);
                    hj = ly.holds + hjrow;
                }
                bool live = act;
                uint32_t gp = NONE32;
                for (uint32_t step = 0; step < SEG_STEPS; step++) {
                    if (!__ballot(live)) break;
                    uint32_t lp = NONE32;
                    if (live) {
                        const uint64_t base = gpos + (uint64_t)sub * PROBE_WORDS;
                        uint4 hv[PROBE_WORDS / 2], nv[PROBE_WORDS / 2];
#pragma unroll
                        for (uint32_t u = 0; u < PROBE_WORDS / 2; u++) {
                            const uint64_t idx = base + 2 * u;
                            if (idx < Ws) {
                                if constexpr (MIRROR) hv[u] = holds_load4(ly.holds, sz.hbytes, hjrow + (uint32_t)idx);
                                else hv[u] = *reinterpret_cast<const uint4 *>(hj + idx);
                                nv[u] = *reinterpret_cast<const uint4 *>(nd + idx);
                            } else {
                                hv[u] = make_uint4(0, 0, 0, 0);
                                nv[u] = make_uint4(0, 0, 0, 0);
                            }
                        }
                        // group steps start past the per-lane probe, above the cursor
#pragma unroll
                        for (int u = (int)(PROBE_WORDS / 2) - 1; u >= 0; u--) {
                            const uint32_t r = first4(and4(hv[u], nv[u]));
                            if (r != NONE32) lp = (uint32_t)base * 64u + 128u * (uint32_t)u + r;
                        }
                    }
                    for (uint32_t off = 1; off < G; off <<= 1) lp = min(lp, (uint32_t)__shfl_xor((int)lp, off));
                    if (live) {
                        if (lp != NONE32) {
                            gp = lp;
                            live = false;
                        } else {
                            gpos += (uint64_t)G * PROBE_WORDS;
                            if (gpos >= Ws) live = false;
                        }
                    }
                }
                if (act && sub == 0) {
                    // word positions these steps passed: through the pick's word, or the probed range
                    ws.seg_p[j] = gp;
                    ws.seg_pos[j] = live ? (uint32_t)gpos : NONE32;
                    ws.pick[j] = (uint32_t)((gp != NONE32 ? (uint64_t)(gp >> 6) + 1 : min(gpos, Ws)) - max(gstart, gw0));
                }
                wave_sync();
                if (scanning) {
                    p = ws.seg_p[lane];
                    scanned += ws.pick[lane];
                    const uint32_t sp = ws.seg_pos[lane];
                    scanning = sp != NONE32;
                    pos = sp;
                }
            }
            acc.lane_words += scanned;
            uint64_t cmask = __ballot(scanning);
            while (cmask) {
                // continue after the probed words (from the cursor when none were probed)
                const int j = __builtin_ffsll((long long)cmask) - 1;
                cmask &= cmask - 1;
                const uint32_t sj = readlane32(ds.src, (uint32_t)j);
                const uint32_t from = max((uint32_t)(readlane64(pos, (uint32_t)j) * 64), ws.cur[j]);
                uint64_t w = 0;
                const uint32_t pj =
                    wave_first_candidate<MIRROR>(ly.holds, sz.hbytes, ly.holds + (uint64_t)sj * Wp, nd, from, Ws, w);
                if ((int)lane == j) p = pj;
                acc.words += w;
            }
            uint32_t pk = NONE32;
            if (mine && md != M_IDLE) {
                pk = min(md == M_FULL ? p : NONE32, ws.xpick[lane]);
                if (pk == NONE32) {
                    md = M_IDLE;
                    ds.idle = 1;
                    ws.cur[lane] = END;
                    ws.known[lane] = 0;
                }
                ws.mode[lane] = md;
            }
            const bool act = mine && md != M_IDLE;
            // (the parts of a split destination decide together, below)
            if (!split && !__ballot(act)) break;
            // clash resolution among d's in-links: fastest link, then lowest id.
            // With few picking links every pick is compared with every other
            // one, read from its lane.  Otherwise picks are hashed into a
            // table of lane ids; a lane alone in its slot has no rival and
            // wins; lanes sharing a slot are grouped by equal pick, and each
            // group keeps its smallest (time, link id).
            const uint64_t actm = __ballot(act);
            const bool few = __popcll(actm) <= FEW_PICKS;
            const uint64_t key = act ? (((uint64_t)ds.tim << 32) | ds.lid) : NONE64;
            const uint32_t hs = act ? (pk * 2654435761u) >> 22 : 0u;
            bool win = act;
            if (few) {
                for (uint64_t m = actm; m; m &= m - 1) {
                    const uint32_t j = (uint32_t)__builtin_ffsll((long long)m) - 1u;
                    if (readlane32(pk, j) == pk && readlane64(key, j) < key) win = false;
                }
            } else {
                if (act) ws.clash_lane[hs] = (uint8_t)lane;
                wave_sync();
                bool rival = false;
                if (act && ws.clash_lane[hs] != lane) {
                    rival = true;
                    ws.clash_hit[hs] = 1;
                }
                wave_sync();
                if (act && ws.clash_hit[hs]) rival = true;
                win = act && !rival;
                uint64_t contested = __ballot(rival);
                if (contested) {
                    wave_sync();
                    if (rival) ws.clash_hit[hs] = 0;
                    while (contested) {
                        const int j = __builtin_ffsll((long long)contested) - 1;
                        const uint32_t v = readlane32(pk, (uint32_t)j);
                        const uint64_t g = __ballot(act && pk == v);
                        const bool in_g = (g >> lane) & 1ull;
                        const uint64_t kmin = wave_min64(in_g ? key : NONE64);
                        if (in_g) win = key == kmin;
                        contested &= ~g;
                    }
                }
            }
            // a split destination's parts publish their winners; every part
            // then finds, for every part's winners, which lose to a winner of
            // another part (same chunk, smaller (time, link id))
            bool group_losers = false;
            if (split) {
                WinTable &tb = win_table(ws);
                const uint64_t wm = __ballot(win);
                if (win) {
                    const uint32_t i = lane_prefix(wm, lane);
                    tb.chunk[i] = pk;
                    tb.tim[i] = ds.tim;
                    tb.lid[i] = ds.lid;
                }
                // (the ballot is taken by the whole wave, not inside the
                // lane-0 branch, where it would see lane 0 alone)
                const uint64_t lost = __ballot(act && !win);
                if (lane == 0) {
                    gs.wcnt[ds.part] = (uint32_t)__popcll(wm);
                    gs.flag[ds.part] = (actm ? 1u : 0u) | (lost ? 2u : 0u);
                }
                __syncthreads();
                bool any_act = false;
                for (uint32_t q = 0; q < ds.nparts; q++) {
                    any_act |= (gs.flag[q] & 1u) != 0;
                    group_losers |= (gs.flag[q] & 2u) != 0;
                }
                if (!any_act) {
                    // nobody picked: the round ends for every part (a
                    // barrier first, so that no part writes its table of the
                    // next round while others read this one's flags)
                    __syncthreads();
                    break;
                }
                uint64_t myfin = 0;
#pragma unroll
                for (uint32_t q = 0; q < NWAVES; q++) {
                    if (q >= ds.nparts) break;
                    const uint32_t nq = gs.wcnt[q];
                    bool ok = lane < nq;
                    if (ok) {
                        const WinTable &a = win_table(grp[q]);
                        const uint32_t c = a.chunk[lane];
                        const uint64_t kq = ((uint64_t)a.tim[lane] << 32) | a.lid[lane];
                        for (uint32_t r = 0; r < ds.nparts && ok; r++) {
                            if (r == q) continue;
                            const WinTable &b = win_table(grp[r]);
                            for (uint32_t i = 0; i < gs.wcnt[r]; i++)
                                if (b.chunk[i] == c && (((uint64_t)b.tim[i] << 32) | b.lid[i]) < kq) ok = false;
                        }
                    }
                    const uint64_t fq = __ballot(ok);
                    if (lane == 0) ws.fin[q] = fq;
                    if (q == ds.part) myfin = fq;
                    group_losers |= fq != (nq >= 64 ? ~0ull : ((1ull << nq) - 1ull));
                }
                if (win) win = (myfin >> lane_prefix(wm, lane)) & 1ull;
            }
            const uint64_t wins = __ballot(win);
            const uint64_t losers = __ballot(act && !win);
            uint32_t ce = 0;
            unsigned long long logq = 0;
            if (split) {
                // this round's slots of the shared send-log segment
                if (lane == 0) ws.logq = wins ? atomicAdd(&gs.log_next, (unsigned long long)__popcll(wins)) : 0ull;
                wave_sync();
                logq = ws.logq;
            }
            bool overflow = false;
            if (act) {
                if (win) {
                    atomicAnd((unsigned long long *)&nd[pk >> 6], ~(1ull << (pk & 63)));
                    const uint64_t end = (uint64_t)t + ds.tim;
                    if (end > 0xFFFFFFFFull) {
                        record_error(ly.ctl, ST_ERANGE, pk, d, 2);
                        overflow = true;
                    }
                    const uint32_t e32 = end > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)end;
                    ds.infl = pk;
                    ds.busy = e32;
                    ds.idle = 0;
                    ds.ready = 0;
                    ds.ready_c = NONE32;
                    ce = e32;
                    __hip_atomic_store(&snap0[sl], ((uint64_t)pk << 32) | e32, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    const unsigned long long q = (split ? logq : ds.log + n_send) + lane_prefix(wins, lane);
                    ly.skey[0][q] = ((uint64_t)t << 32) | ds.lid;
                    ly.sval[0][q] = pk;
                    const uint32_t kn = ws.known[lane];
                    ws.known[lane] = kn ? kn - 1u : 0u;  // pk was one of its candidates
                    if (md == M_FULL) {
                        ws.cur[lane] = pk + 1;
                        md = M_IDLE;
                    } else {
                        ws.cur[lane] = END;
                        md = M_ARR_WON;
                    }
                } else if (md == M_FULL) {
                    ws.cur[lane] = pk + 1;
                }
                ws.mode[lane] = md;
            }
            n_send += (uint32_t)__popcll(wins);
            acc.clashes += (unsigned long long)__popcll(losers);
            acc.lane_cstar = max(acc.lane_cstar, ce);
            if (__ballot(overflow)) acc.err = 1;
            wave_sync();
            // a candidate found ahead of time is gone once its chunk is
            // delivered.  With few picks it is compared with the winners'
            // picks; otherwise winners stamp their chunk's hash slot with the
            // round, and a stamped slot drops the candidate (a hash collision
            // only drops one that is still valid, which costs a scan)
            if (split) {
                // every part's winners, from their tables
#pragma unroll
                for (uint32_t q = 0; q < NWAVES; q++) {
                    if (q >= ds.nparts) break;
                    const WinTable &a = win_table(grp[q]);
                    for (uint64_t m = ws.fin[q]; m; m &= m - 1) {
                        const uint32_t c = a.chunk[__builtin_ffsll((long long)m) - 1];
                        if (c == ds.ready_c) ds.ready_c = NONE32;
                    }
                }
                if (n_arr | n_unf) {
#pragma unroll
                    for (uint32_t q0 = 0; q0 < NWAVES; q0++) {
                        if (q0 >= ds.nparts) break;
                        const WinTable &a = win_table(grp[q0]);
                        for (uint64_t m = ws.fin[q0]; m; m &= m - 1) {
                            const uint32_t c = a.chunk[__builtin_ffsll((long long)m) - 1];
                            for (uint32_t q = lane; q < n_arr; q += 64)
                                if (ws.arr_c[q] == c) ws.arr_need[q] = 0;
                            for (uint32_t q = lane; q < n_unf; q += 64)
                                if (ws.unf_c[q] == c) ws.unf_need[q] = 0;
                        }
                    }
                }
            } else if (few) {
                bool gone = false;
                for (uint64_t m = wins; m; m &= m - 1)
                    gone |= readlane32(pk, (uint32_t)__builtin_ffsll((long long)m) - 1u) == ds.ready_c;
                if (gone) ds.ready_c = NONE32;
            } else {
                if (win) ws.dlv_round[hs] = (uint16_t)acc.rounds;
                wave_sync();
                if (ds.ready_c != NONE32 && ws.dlv_round[(ds.ready_c * 2654435761u) >> 22] == (uint16_t)acc.rounds)
                    ds.ready_c = NONE32;
            }
            // the delivered chunks are no longer needed: clear their flags
            // (each entry is compared with the winners' picks, read from
            // their lanes)
            // (wave-uniform loops: the winners' picks are read lane by lane)
            if (!split && (n_arr | n_unf) && wins) {
                for (uint32_t q0 = 0; q0 < n_arr; q0 += 64) {
                    const uint32_t q = q0 + lane;
                    const uint32_t c = q < n_arr ? ws.arr_c[q] : NONE32;
                    bool hit = false;
                    for (uint64_t wm = wins; wm; wm &= wm - 1)
                        hit |= readlane32(pk, (uint32_t)__builtin_ffsll((long long)wm) - 1u) == c;
                    if (hit) ws.arr_need[q] = 0;
                }
                for (uint32_t q0 = 0; q0 < n_unf; q0 += 64) {
                    const uint32_t q = q0 + lane;
                    const uint32_t c = q < n_unf ? ws.unf_c[q] : NONE32;
                    bool hit = false;
                    for (uint64_t wm = wins; wm; wm &= wm - 1)
                        hit |= readlane32(pk, (uint32_t)__builtin_ffsll((long long)wm) - 1u) == c;
                    if (hit) ws.unf_need[q] = 0;
                }
            }
            wave_sync();
            // a link that won an arrival keeps the other arrivals as its cursor
            if (__ballot(md == M_ARR_WON)) {
                for (uint32_t q = lane; q < n_arr; q += 64) {
                    if (ws.arr_end[q] != t || !ws.arr_need[q]) continue;
                    const uint32_t j = ws.arr_j[q];
                    if (ws.mode[j] == M_ARR_WON) atomicMin(&ws.cur[j], ws.arr_c[q]);
                }
                wave_sync();
                if (md == M_ARR_WON) {
                    md = M_IDLE;
                    ws.mode[lane] = md;
                }
            }
            if (!split || ds.part == 0) acc.rounds++;
            wave_sync();
            if (split) {
                // the round's commits (needs row) are seen by every part's
                // next picks, and nobody writes a table still being read
                if constexpr (!MIRROR) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): needs row in device memory
                __syncthreads();
                if (!group_losers) break;
            } else if (!losers) {
                // no loser: every link that picked has committed, and a
                // further round would find no link left to pick
                break;
            }
        }
        t_prev = t;
    }

    // a resident wave issues the look-ahead after the window exchange is
    // published (look_ahead_late), so the publish does not wait for it
    if (!resident) look_ahead_issue<MIRROR>(ly, sz.hbytes, Wp, Ws, ws, ds, nd, mine, n_arr, n_unf, la);
    ds.n_arr_prev = n_arr;
    ds.n_unf_prev = n_unf;
    if (!resident) look_ahead_finish<MIRROR>(Ws, ws, ds, nd, mine, la);
    acc.tmin = min(acc.tmin, wave_min(mine && ds.infl != NONE32 ? ds.busy : NONE32));
    ds.log += n_send;
    acc.sent += n_send;
    wave_sync();
}

// The look-ahead of a resident wave, issued once its workgroup has published
// the window: its loads travel during the exchange instead of delaying the
// publish.  Holds rows read this late hold at most the arrivals of the window
// just ended beyond what they held at its end (other workgroups fold those at
// the start of the next window), and the window's arrival lists, which the
// look-ahead adds, contain them already; so the result is the same.
template <bool MIRROR>
__device__ __forceinline__ void look_ahead_late(const Layout &ly, const Sizes &sz, const WaveShared &ws,
                                                const Dest &ds, LookAhead &la)
{
    if (ds.n == 0) return;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t Wp = sz.Wp, Ws = (sz.W + 1) & ~1ull;
    const uint64_t *nd;
    if constexpr (MIRROR) nd = needs_lds + (uint64_t)((threadIdx.x >> 6) - ds.part) * Wp;  // part 0's row
    else nd = ly.needs + (uint64_t)ds.d * Wp;
    look_ahead_issue<MIRROR>(ly, sz.hbytes, Wp, Ws, ws, ds, nd, lane < ds.n, ds.n_arr_prev, ds.n_unf_prev, la);
}

// MIRROR: every wave owns one destination for the whole run and keeps its
// needs row in LDS (the host checks both).  SPLIT: some destinations are
// split over the waves of a workgroup (a separate build of the kernel, so
// that the others carry none of the part synchronisation; it needs every
// wave resident, so the build that keeps needs rows in device memory is
// held to two workgroups per compute unit, spilling registers, to keep one
// wave per destination on the largest topologies).
template <bool MIRROR, bool SPLIT>
__global__ void __launch_bounds__(NT, (!MIRROR && SPLIT) ? 2 : 1) k_match(Layout ly, Sizes sz)
{
    __shared__ BlockShared sh;
    Control *ctl = ly.ctl;
    if (__hip_atomic_load(&ctl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    // queued next to the switch-group kernel: runs only when the check found
    // that the no-multicast rule cannot act
    if (sz.sw_gate && __hip_atomic_load(&ctl->sw_binds, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    const uint32_t tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t wpb = blockDim.x >> 6;  // waves in this workgroup (1..NWAVES)
    const uint32_t gwave = blockIdx.x * wpb + wave, nwaves = gridDim.x * wpb;
    if (ctl->needs_total == 0) {
        if (blockIdx.x == 0 && tid == 0) ctl->windows = 0;
        return;
    }
    const unsigned long long max_windows = ctl->needs_total + 2ull;
    // every wave owns at most one destination (or part of one): its state
    // stays on chip
    const bool resident = sz.resident != 0;
    // (the host picks the kernels with needs rows in LDS or with split
    // destinations only with one destination per wave, and the first only
    // with a holds bitmap the buffer descriptor spans)
    if ((MIRROR && (!resident || sz.hbytes == 0)) || (SPLIT && !resident)) {
        if (blockIdx.x == 0 && tid == 0) record_error(ctl, ST_EINTERNAL, 2, 0, 0);
        return;
    }
    WaveShared &ws = sh.w[wave];
    Dest ds{};
    for (uint32_t i = lane; i < CLASH_SLOTS; i += 64) {
        ws.clash_hit[i] = 0;
        ws.dlv_round[i] = 0xFFFFu;
    }
    const uint32_t passes = (sz.D + nwaves - 1) / nwaves;
    const uint32_t mine_d = resident ? ly.wave_dest[gwave] : NONE32;
    if (mine_d != NONE32) load_dest(ly, ws, mine_d, ly.wave_part[gwave], ds);
    // a split destination's send-log segment is shared by its parts
    if (SPLIT && mine_d != NONE32 && ds.nparts > 1 && ds.part == 0 && lane == 0) sh.g.log_next = ds.log;
    if constexpr (MIRROR) {
        if (mine_d != NONE32 && ds.part == 0) {
            uint64_t *row = needs_lds + (uint64_t)wave * sz.Wp;
            const uint64_t *g = ly.needs + (uint64_t)mine_d * sz.Wp;
            for (uint64_t i = 2 * lane; i < sz.Wp; i += 128)
                *reinterpret_cast<uint4 *>(row + i) = *reinterpret_cast<const uint4 *>(g + i);
        }
        wave_sync();
    }
    // the parts of a split destination see part 0's row and log slot
    if constexpr (SPLIT) __syncthreads();
    Acc acc = {NONE32, 0u, 0u, 0ull, 0ull, 0ull, 0ull, 0ull, 0u};
    LookAhead la;
    la.cur = NONE32;
    la.n_arr = la.n_unf = 0;
    la.words = 0;
    unsigned long long remaining = ctl->needs_total;
    uint32_t t0 = 0;
    unsigned long long k = 0;
    for (;; k++) {
        const uint64_t t1 = (uint64_t)t0 + sz.tmin;
        acc.tmin = NONE32;
        const unsigned long long sent0 = acc.sent;
        if (resident) {
            if (mine_d != NONE32)
                process_window<MIRROR, SPLIT>(ly, sz, ws, ds, (uint32_t)k, t0, t1, true, acc, la, sh.w + (wave - ds.part),
                                              sh.g);
        } else if constexpr (!MIRROR) {
            for (uint32_t r = 0; r < passes; r++) {
                const uint32_t d = ly.wave_dest[(uint64_t)r * nwaves + gwave];
                if (d == NONE32) continue;
                load_dest(ly, ws, d, 0u, ds);
                process_window<false, false>(ly, sz, ws, ds, (uint32_t)k, t0, t1, false, acc, la, sh.w, sh.g);
                store_dest(ly, ws, ds);
            }
        }
        if (lane == 0) {
            sh.red_tmin[wave] = acc.tmin;
            sh.red_err[wave] = acc.err;
            sh.red_sent[wave] = acc.sent - sent0;
        }
        // the window's writes and atomics of this wave are performed before
        // the barrier, so the slot written after it publishes all of them
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        __syncthreads();
        uint32_t bmin = NONE32, berr = 0;
        unsigned long long bsent = 0;
        for (uint32_t w = 0; w < wpb; w++) {
            bmin = min(bmin, sh.red_tmin[w]);
            berr |= sh.red_err[w];
            bsent += sh.red_sent[w];
        }
        Exchange ex;
        window_publish(ly.xslot, (uint32_t)k, bmin, bsent, berr);
        if (resident && mine_d != NONE32) {
            look_ahead_late<MIRROR>(ly, sz, ws, ds, la);
            // waves that do not poll the exchange finish it while they wait
            // (it reads nothing the exchange changes); the call at the next
            // window's start then finds nothing left to do
            if (wave != wpb - 1u && ds.n > 0) {
                const uint64_t *nd;
                if constexpr (MIRROR) nd = needs_lds + (uint64_t)(wave - ds.part) * sz.Wp;  // part 0's row
                else nd = ly.needs + (uint64_t)ds.d * sz.Wp;
                look_ahead_finish<MIRROR>((sz.W + 1) & ~1ull, ws, ds, nd, lane < ds.n, la);
            }
        }
        if (!window_wait<MIRROR>(ctl, ly.xslot, sh, (uint32_t)k, ex)) break;
        remaining -= ex.sent;
        if (ex.err || remaining == 0) break;
        if (ex.tn == NONE32) {
            record_error(ctl, ST_EDEADLOCK, (uint32_t)remaining, 0, 0);
            break;
        }
        if (k + 1 >= max_windows) {
            record_error(ctl, ST_EINTERNAL, 1, 0, 0);
            break;
        }
        t0 = ex.tn;
    }
    if (blockIdx.x == 0 && tid == 0) {
        ctl->needs_remaining = remaining;
        ctl->windows = k + 1;
        ctl->n_log = ctl->needs_total - remaining;
    }
    acc.words += wave_sum64(acc.lane_words + la.words);
    acc.cstar = max(acc.cstar, wave_max(acc.lane_cstar));
    if (lane == 0) {
        atomicMax(&ctl->cstar, acc.cstar);
        if (acc.clashes) atomicAdd(&ctl->clashes, acc.clashes);
        if (acc.rounds) atomicAdd(&ctl->rounds, acc.rounds);
        if (acc.words) atomicAdd(&ctl->scan_words, acc.words);
    }
}

}  // namespace

namespace {
const void *match_kernel(bool mirror, bool split)
{
    if (split)
        return mirror ? reinterpret_cast<const void *>(k_match<true, true>)
                      : reinterpret_cast<const void *>(k_match<false, true>);
    return mirror ? reinterpret_cast<const void *>(k_match<true, false>) : reinterpret_cast<const void *>(k_match<false, false>);
}
}  // namespace

size_t match_static_lds()
{
    hipFuncAttributes a{};
    if (hipFuncGetAttributes(&a, match_kernel(true, false)) != hipSuccess) return 0;
    return a.sharedSizeBytes;
}

int match_max_grid(int device, int waves_per_block, bool mirror, size_t dyn_lds, bool split)
{
    int per_cu = 0, cus = 0;
    const void *kern = match_kernel(mirror, split);
    if (dyn_lds && hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn_lds) != hipSuccess)
        return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 64 * waves_per_block, dyn_lds) != hipSuccess)
        return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) return 0;
    return per_cu * cus;
}

hipError_t launch_match(const Layout &ly, const Sizes &sz, hipStream_t st, int grid, int waves_per_block, bool mirror,
                        bool split)
{
    if (waves_per_block < 1 || waves_per_block > (int)NWAVES) return hipErrorInvalidValue;
    const size_t dyn = mirror ? (size_t)waves_per_block * sz.Wp * sizeof(uint64_t) : 0;
    const void *kern = match_kernel(mirror, split);
    if (dyn) {
        const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
        if (e != hipSuccess) return e;
    }
    Layout l = ly;
    Sizes s = sz;
    void *args[] = {&l, &s};
    return hipLaunchCooperativeKernel(kern, dim3(grid), dim3(64 * waves_per_block), args, dyn, st);
}

}  // namespace pccl
