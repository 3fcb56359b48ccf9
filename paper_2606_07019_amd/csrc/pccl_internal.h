// Internal definitions of the MI355X synthesis matcher (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pccl {

constexpr uint32_t NONE32 = 0xFFFFFFFFu;
constexpr uint64_t NONE64 = 0xFFFFFFFFFFFFFFFFull;

// Row padding of the chunk bitmaps: 128 words (1 KiB), one wave64 sweep of
// 16-byte loads, so a sweep never needs a tail check inside a row.
constexpr uint32_t ROW_ALIGN_WORDS = 128;

// Matching kernel envelope (checked on the host when a topology is loaded).
constexpr uint32_t MATCH_THREADS = 256;   // at most 4 wavefronts per workgroup (one per SIMD), one destination device each
constexpr uint32_t MATCH_WAVES = MATCH_THREADS / 64;
constexpr uint32_t MAX_IN_LINKS = 64;     // in-links of one wave's part of a device (one lane each)
constexpr uint32_t MAX_PAIRS = 512;       // sum over a wave's in-links of their sources' in-degree
// A device with more in-links or arrival pairs than one wave takes is split
// over the waves of one workgroup (each wave one part of its in-links).
constexpr uint32_t MAX_SPLIT_LINKS = MATCH_WAVES * MAX_IN_LINKS;
constexpr uint32_t MAX_DEVICES_SP = 8000; // shortest paths keep one 64-bit distance per device in LDS
static_assert(MAX_DEVICES_SP <= 0xFFFF, "switch-group tables hold device ids in 16 bits");
constexpr uint32_t MAX_MATCH_GRID = 1024; // workgroups of the matching kernel (window exchange slots)
constexpr uint32_t MATCH_TARGET_GRID = 128; // workgroups the matching kernel aims for (measured on MI355X)
constexpr uint32_t XSLOT_WORDS = 16;        // one 128-byte line per window exchange slot

// Switch-model matching kernel envelope (one workgroup owns a switch group:
// a switch with its out-neighbours; checked on the host).
// 768 threads: three waves per SIMD, so a wave may hold 168 registers
// (with four waves, 128 were not enough for the pick stage).
constexpr uint32_t SW_THREADS = 768;
constexpr uint32_t SW_MAX_LINKS = 768;   // in-links of the destinations of one group
constexpr uint32_t SW_MAX_SRC = 768;     // distinct sources of those links
constexpr uint32_t SW_MAX_PAIRS = 6144;  // in-links of those sources (arrival slots)
constexpr uint32_t SW_MAX_SW = 64;       // unicast or limited switches in one group
constexpr uint32_t SW_MAX_SRC_IN = 64;   // in-links of one source of a group link (one bit each in a link's arrival mask)
constexpr uint32_t SW_MAX_POOL = 1024;   // buffer places of a group's limited switches
constexpr uint8_t SW_NONE8 = 0xFF;

// Status codes mirrored from the public header.
enum : uint32_t {
    ST_OK = 0, ST_EINVAL = 1, ST_EUNREACHABLE = 2, ST_ERANGE = 3, ST_ENOMEM = 4,
    ST_EDEVICE = 5, ST_ESTATE = 6, ST_EUNSUPPORTED = 7, ST_EDEADLOCK = 8, ST_EINTERNAL = 9
};

// Device-side control block: error reporting, counters, window bookkeeping.
struct Control {
    uint32_t error;          // first error code recorded (0 = none)
    uint32_t error_arg[3];   // chunk / device / detail of the first error
    unsigned long long needs_total;      // (device, chunk) deliveries required
    unsigned long long needs_remaining;  // still undelivered
    unsigned long long n_log;            // sends logged so far
    unsigned long long max_sends;        // capacity of the send log
    unsigned long long rounds, clashes, windows;
    unsigned long long scan_words;       // words of each row read by the intersect
    uint32_t n_sources;      // distinct chunk sources
    uint32_t abort;          // set when a window exchange wait times out
    uint32_t cstar;          // collective time of the copy schedule
    uint32_t sort_cur;       // radix sort: buffer holding the current order
    uint32_t sort_buf[9];    // radix sort: buffer holding the order before pass i of a sort
    uint32_t sort_skip;      // radix sort (scan kernel): the pending pass is a no-op
    uint32_t sw_binds;       // switch model: the no-multicast rule can change the schedule
};

__device__ inline void record_error(Control *ctl, uint32_t code, uint32_t a = 0, uint32_t b = 0,
                                    uint32_t c = 0)
{
    if (atomicCAS(&ctl->error, 0u, code) == 0u) {
        ctl->error_arg[0] = a;
        ctl->error_arg[1] = b;
        ctl->error_arg[2] = c;
    }
}

__device__ inline uint64_t splitmix64_key(uint64_t seed, uint64_t c)
{
    // Output number c+1 of SplitMix64 started at state `seed`
    // (Steele, Lea and Flood, "Fast splittable pseudorandom number
    // generators", OOPSLA 2014): golden-gamma increment, then the
    // variant-13 finalizer of the MurmurHash3 mixer.
    uint64_t z = seed + (c + 1ull) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Tables of the switch-model matching kernel, built on the host (one u32
// region of the workspace).  Group g's header sits at grp[16 g]: link
// count and base, destination count and base, source count and base, arrival
// pair count and base, unicast switch count and base, unicast out-link list
// base, limited switch count and base, out-neighbour list base, buffer pool
// base and size.  Per-group arrays are indexed base + local index.
struct SwTab {
    const uint32_t *grp;      // [16 G]
    const uint32_t *blk;      // [nb + 1] groups of workgroup b: blk_list[blk[b] .. blk[b+1])
    const uint32_t *blk_list; // [G]
    const uint32_t *lk_slot;  // destination-major slot of each group link
    const uint32_t *lk_dl;    // its destination's index in the group
    const uint32_t *lk_srcj;  // its source's index in the group's source list
    const uint32_t *lk_uni;   // group index of its source if a unicast switch, else NONE32
    const uint32_t *lk_dbuf;  // group index of its destination if a limited switch, else NONE32
    const uint32_t *lk_sbuf;  // group index of its source if a limited switch, else NONE32
    const uint32_t *d_off;    // [nD + 1] per group: links of destination dl
    const uint32_t *s_poff;   // [nS + 1] per group: arrival pairs of source j
    const uint32_t *p_slot;   // group link position of each pair's link (an in-link of the source)
    const uint32_t *u_off;    // [nU + 1] per group: out-links of unicast switch u
    const uint32_t *u_list;   // group-local link indices
    const uint32_t *b_cap;    // [nB + 1] per group: buffer capacity of limited switch b
    const uint32_t *b_poff;   // [nB + 1] per group: its places in the group's pool
    const uint32_t *b_ooff;   // [nB + 1] per group: its out-neighbours
    const uint32_t *b_out;    // out-neighbours: device id (low 16 bits), group destination index (high 16)
    const uint32_t *uc_off;   // [n_uni + 1] every unicast switch of the model: its out-neighbours in uc_dst
    const uint32_t *uc_dst;   // out-neighbour device ids
    const uint32_t *b_abs;    // [2 nBt] per limited-switch row (group's bbase + b): first out-neighbour in b_out, count
    uint32_t *pool_c, *pool_n;  // buffer places: chunk, out-neighbours still needing it (0 = free)
    uint32_t *occ;              // [nB + 1] per group: occupied places
    uint32_t *acnt;             // [nBt C] per limited-switch row and chunk rank: out-links whose destination still needs it
};

// Pointers into the caller's workspace (all device memory).
struct Layout {
    // topology, link order
    uint32_t *lsrc, *ldst, *ltime, *lrev;
    // topology, destination-major "slot" order (in-links grouped by destination)
    uint32_t *in_off;      // [D+1]
    uint32_t *slot_link;   // [L] link id of slot
    uint32_t *slot_src;    // [L] source device of slot
    uint32_t *slot_time;   // [L]
    uint32_t *slot_cum;    // [L] prefix of source in-degrees inside the destination
    uint32_t *dest_pairs;  // [D] total of source in-degrees over the destination's in-links
    uint64_t *group_masks; // [G * WN]
    // the collective's inputs, copied in from the context's host staging
    uint64_t *pre, *post;  // [N * W] each, the caller's bitmap layout
    uint16_t *chunk_group; // [C], null with one group
    // chunk setup
    uint32_t *chunk_src;   // [C]
    uint32_t *holder_cnt;  // [C] bit 31: has a postcondition bit
    uint64_t *chunk_dist;  // [C]
    uint32_t *rank;        // [C] chunk -> priority position
    uint32_t *order;       // [C] priority position -> chunk
    uint32_t *src_index;   // [N] row of a source in the shortest-path tables
    uint32_t *src_list;    // [N]
    uint64_t *sp_dist;     // [N * D]
    uint32_t *sp_parent;   // [N * D]
    // sort buffers (chunk order first, then the send log)
    uint64_t *skey[2];     // [max(C, 2*max_sends)]
    uint32_t *sval[2];
    uint32_t *hist;        // [256 * hist_stride(max_tiles)]: tile-major 32-bit or digit-major 16-bit counts
    // matching state
    uint64_t *holds, *needs;  // [D * Wp]
    uint32_t *busy, *infl, *cur, *lflags;  // [L] by slot
    uint32_t *lcnt;           // [L] by slot: bound on the link's candidates (source holds, destination needs)
    uint64_t *snap;           // [3 * L] by slot
    unsigned long long *dest_log;  // [D] next send-log slot of each destination
    uint64_t *xslot;          // [2 * MAX_MATCH_GRID * XSLOT_WORDS] window exchange slots of the matching kernel
    uint32_t *wave_dest;      // [D + MATCH_WAVES * MAX_MATCH_GRID] destination of (pass, wave), NONE32 if none
    uint32_t *wave_part;      // [same] for a split destination: parts << 24 | part << 16 | first link << 8 | links; 0 = whole
    SwTab sw;                 // switch-model tables (null pointers without a switch model)
    // output
    void *out;                // pccl_send [2 * max_sends]
    Control *ctl;
};

struct Sizes {
    uint32_t N, S, D, L, C, G;
    uint64_t W;    // words per chunk row of the caller's pre/post bitmaps
    uint64_t Wp;   // padded words per row of the device bitmaps
    uint64_t WN;   // words per group mask
    uint64_t max_sends;
    uint32_t tmin; // smallest link time (window length)
    uint32_t max_tiles;
    uint32_t hbytes;  // bytes of the holds bitmap (D rows of Wp words) when below 2 GiB, else 0
    uint32_t resident; // every wave of the matching kernel owns one destination (or part) for the whole run
    uint32_t sw_gate;  // both matching kernels are queued; Control::sw_binds picks the one that runs
    uint32_t sw_nbt;   // limited-switch rows of the switch tables (0: no switch model or no limited switch)
};

// ---- launchers (each defined in the translation unit that holds its kernels)
hipError_t launch_setup(const Layout &ly, const Sizes &sz, const uint64_t *pre, const uint64_t *post,
                        const uint16_t *chunk_group, uint64_t seed, hipStream_t st);
// mirror: every wave keeps its destination's needs row in LDS (waves_per_block
// rows of Wp words of dynamic shared memory); requires one destination per wave.
// split: some destinations are split over the waves of a workgroup (the
// kernel variants with part synchronisation)
hipError_t launch_match(const Layout &ly, const Sizes &sz, hipStream_t st, int grid, int waves_per_block, bool mirror,
                        bool split);
int match_max_grid(int device, int waves_per_block, bool mirror, size_t dyn_lds, bool split);
size_t match_static_lds();  // static LDS bytes of the matching kernel
hipError_t launch_match_sw(const Layout &ly, const Sizes &sz, hipStream_t st, int grid);
// sets Control::sw_binds when two out-neighbours of one of the n_uni unicast
// switches need the same chunk
hipError_t launch_unicast_check(const Layout &ly, const Sizes &sz, hipStream_t st, uint32_t n_uni);
int match_sw_max_grid(int device);
hipError_t launch_output(const Layout &ly, const Sizes &sz, int op, uint64_t n, hipStream_t st);
// LSD radix sort of (key, value) pairs by key bytes [byte_lo, byte_hi), stable;
// the sorted order ends up in buffer ly.ctl->sort_cur (read it on the device).
// time_gate: the bytes are start-time bytes (key bits 32..63) and a byte
// past the device's collective time is skipped.
hipError_t radix_sort_pairs(const Layout &ly, uint64_t n, int byte_lo, int byte_hi, uint32_t max_tiles,
                            bool reset_cur, hipStream_t st, bool time_gate = false);
constexpr uint32_t SORT_TILE = 4096;      // elements per radix-sort tile
constexpr uint32_t SORT_THREADS = 256;
// row length of the digit-major tile histogram, 16-bit counts (a multiple
// of 8 tiles, so a row is read in 16-byte loads)
inline __host__ __device__ uint32_t hist_stride(uint32_t tiles) { return (tiles + 7u) & ~7u; }

}  // namespace pccl
