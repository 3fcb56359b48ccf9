/*
 * pccl.h -- C ABI of the MI355X synthesis matcher for PCCL
 * ("PCCL: Process Group-Aware Scalable and Generic Collective Algorithm
 * Synthesizer").
 *
 * The library synthesizes a collective algorithm -- a schedule of
 * (link, chunk, start time) transfers -- for a modeled network topology, a
 * collective given as NPU-centric pre/postconditions, and one or more process
 * groups.  Everything from the derivation of the conditions to the canonical
 * schedule runs on one AMD Instinct GPU (gfx950); the host side only checks
 * and stages the small topology arrays and launches kernels.
 *
 * Call order: pccl_create -> pccl_load_topology -> [pccl_set_switch_model]
 * -> pccl_set_collective -> pccl_workspace_bytes -> pccl_set_workspace ->
 * pccl_synthesize (any number of times) -> pccl_get_schedule / pccl_get_stats / pccl_get_setup ->
 * pccl_destroy.  A call made out of order returns PCCL_ESTATE.  A context is
 * not thread-safe; use one per thread.
 *
 * Every function returns a pccl_status; no C++ exception crosses the ABI.
 * pccl_last_error() returns a message for the last failed call.
 */
#ifndef PCCL_H
#define PCCL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pccl_ctx pccl_ctx;

typedef enum {
    PCCL_OK = 0,
    PCCL_EINVAL = 1,        /* malformed topology or collective */
    PCCL_EUNREACHABLE = 2,  /* a destination cannot be reached from its source */
    PCCL_ERANGE = 3,        /* a time in ns does not fit in 32 bits */
    PCCL_ENOMEM = 4,        /* workspace too small for this collective */
    PCCL_EDEVICE = 5,       /* a HIP call failed */
    PCCL_ESTATE = 6,        /* call out of order */
    PCCL_EUNSUPPORTED = 7,  /* outside the supported envelope (see each call) */
    PCCL_EDEADLOCK = 8,     /* needs remain but nothing is in flight (never on valid input) */
    PCCL_EINTERNAL = 9      /* internal error (watchdog, caught exception) */
} pccl_status;

/*
 * Collective operations (paper Sec. 4.5, "Reduction Operations").
 *   PCCL_OP_COPY: non-reduction patterns (All-Gather, All-to-All(v),
 *     Broadcast, Scatter, any generic pre/postcondition).
 *   PCCL_OP_REDUCE_REVERSED: pre/post describe the dual copy pattern (e.g.
 *     All-Gather for Reduce-Scatter, Broadcast for Reduce); the output is the
 *     time reversal of the copy schedule: each send (l, c, t) becomes
 *     (reverse(l), c, C* - t - T[l]) with the reduce flag, C* being the copy
 *     schedule's collective time.  Every link needs a reverse link of equal
 *     transfer time, else PCCL_EUNSUPPORTED.
 *   PCCL_OP_ALLREDUCE: pre/post describe the All-Gather half; the output is
 *     the reversed schedule (Reduce-Scatter) followed by the copy schedule
 *     shifted by C*; collective time 2 C*.
 */
typedef enum {
    PCCL_OP_COPY = 0,
    PCCL_OP_REDUCE_REVERSED = 1,
    PCCL_OP_ALLREDUCE = 2
} pccl_op;

/* One transfer of the schedule: `link` starts sending chunk `chunk` (the
 * caller's chunk id) at `t_start_ns`; it occupies the link for T[link] ns.
 * flags bit 0 = the receiver reduces (adds) instead of copying. */
typedef struct {
    uint32_t link;
    uint32_t chunk;
    uint32_t t_start_ns;
    uint32_t flags;
} pccl_send;

#define PCCL_SEND_REDUCE 1u

/* One step of an exported program (pccl_export_program). */
typedef struct {
    uint32_t rank;       /* NPU that executes the step */
    uint32_t tb;         /* thread block of that rank */
    uint32_t op;         /* PCCL_STEP_SEND / PCCL_STEP_RECV / PCCL_STEP_RECV_REDUCE */
    uint32_t peer;       /* the NPU at the other end of the transfer */
    uint32_t chunk;      /* the caller's chunk id */
    uint32_t t_start_ns; /* scheduled start of the transfer */
    uint32_t dep_first;  /* this step waits for deps[dep_first .. dep_first + dep_count) (step indices) */
    uint32_t dep_count;
} pccl_step;

#define PCCL_STEP_SEND 0u
#define PCCL_STEP_RECV 1u
#define PCCL_STEP_RECV_REDUCE 2u

/*
 * Creates a context bound to HIP device `hip_device`.  `tie_seed` seeds the
 * tie-break among chunks of equal distance: chunks are ordered by distance
 * descending (Alg. 3 sorts conditions by their distance, Sec. 4.4), then by
 * the SplitMix64 output number c+1 of a generator started at `tie_seed`
 * ascending.  Returns PCCL_EDEVICE if the device cannot be selected.
 */
pccl_status pccl_create(pccl_ctx **out, int hip_device, uint64_t tie_seed);

/* Releases the context (not the caller's workspace).  NULL is ignored. */
void pccl_destroy(pccl_ctx *ctx);

/*
 * Loads the network (paper Sec. 4.2 TEN; Sec. 4.6 alpha-beta links; Sec. 4.7
 * switches).  Devices 0..n_npus-1 are NPUs, n_npus..n_npus+n_switches-1 are
 * switches (relay-only devices).  Link l is directed link_src[l] ->
 * link_dst[l] with latency alpha_ns[l] and bandwidth bw_GBps[l] (1 GB/s is one
 * byte per ns).  All arrays are host memory of n_links entries and are copied.
 * PCCL_EINVAL: endpoint out of range, self loop, duplicate (src, dst) pair,
 * zero bandwidth, n_npus == 0.  PCCL_EUNSUPPORTED: more than 8000 devices
 * (NPUs plus switches), more than 256 in-links on one device, a device with
 * more than 512 in-links that feeds another, or a device whose in-links'
 * sources have more than 2048 in-links in total.  (The matching kernel gives
 * a device one wavefront, one lane per in-link and lists of up to 512
 * arrival pairs in LDS; a device beyond 64 in-links or 512 pairs is split
 * over the wavefronts of a workgroup of its own, at most four.
 * pccl_set_collective returns PCCL_EUNSUPPORTED when the matching kernel
 * cannot keep a workgroup per split device and a wavefront per other device
 * resident at once: with needs rows too wide for LDS that is 512 workgroups
 * of four wavefronts on MI355X (128 nodes of 8 NPUs behind 128-port switches
 * take 8 + 256 of them).)
 */
pccl_status pccl_load_topology(pccl_ctx *ctx, uint32_t n_npus, uint32_t n_switches,
                               uint32_t n_links, const uint32_t *link_src,
                               const uint32_t *link_dst, const uint32_t *alpha_ns,
                               const uint32_t *bw_GBps);

/*
 * Sets the collective (paper Sec. 2.1 pre/postconditions, Sec. 2.2 process
 * groups, Sec. 4.1 conditions).
 *   n_chunks, chunk_bytes: C chunks of m bytes each (m >= 1).
 *   pre_bits, post_bits: n_npus rows of ceil(C/64) uint64 words, LSB first
 *     (chunk c is bit c%64 of word c/64), in host or device memory.  Row v
 *     of pre holds the chunks NPU v has before the collective, row v of post
 *     the chunks it must have after.
 *   group_masks: HOST pointer to n_groups rows of ceil(n_npus/64) words, the
 *     members of each process group.
 *   chunk_group: C uint16 group ids (host or device memory), or NULL when
 *     n_groups == 1.
 * Every array is copied before the call returns (the bitmaps into pinned
 * host memory the context owns, uploaded to the workspace by the next
 * synthesize call), so the caller may free or reuse them at once.  The call
 * also plans the device work (matching-kernel launch shape, destination
 * deal, switch tables); pccl_set_switch_model re-plans by itself when it
 * comes after.  A previously bound workspace must be bound again.
 * Checked here: sizes and group masks (PCCL_EINVAL); PCCL_EDEVICE if a
 * copy fails.  Checked on the device by pccl_synthesize (PCCL_EINVAL): each
 * chunk with a postcondition bit has exactly one precondition holder, no
 * chunk has two holders, pre/post bits only at members of the chunk's group,
 * no bits beyond chunk C-1, group ids in range.  A link time
 * alpha + ceil(m / bw) above 2^32-1 gives PCCL_ERANGE.
 */
pccl_status pccl_set_collective(pccl_ctx *ctx, uint32_t n_chunks, uint64_t chunk_bytes,
                                const uint64_t *pre_bits, const uint64_t *post_bits,
                                const uint64_t *group_masks, uint32_t n_groups,
                                const uint16_t *chunk_group, pccl_op op);

/*
 * Explicit switch nodes (paper Sec. 4.7, "Modeling Switches"): buffer limits
 * and switches without multicast.  Optional; call after pccl_load_topology
 * (which clears the model) and before pccl_workspace_bytes /
 * pccl_set_workspace (the model changes the workspace; a workspace set
 * earlier must be set again: PCCL_ESTATE until then).
 *   n_switches: must equal the topology's switch count.
 *   buffer_chunks: HOST pointer to n_switches uint32 (copied), or NULL for
 *     all unlimited.  Entry i belongs to device n_npus + i: 0 = unlimited,
 *     else the most chunks the switch buffers at once.  A chunk is buffered
 *     at switch w from the start of its transfer into w until no
 *     out-neighbour of w still needs it; a transfer into w starts only while
 *     fewer chunks than the capacity are buffered there.  Transfers into w
 *     that win their clashes at the same instant take the free places in
 *     (link time, link id) order; the others wait.
 *   unicast: HOST pointer to n_switches uint8 (copied), or NULL for all
 *     multicast.  1 = the switch keeps at most one copy of a chunk in flight
 *     on its out-links (it forwards a chunk to its next neighbours one by
 *     one); out-links of such a switch that pick the same chunk at the same
 *     instant clash, after the destination clash, fastest link first, then
 *     the lowest link id.
 * A model with no limit leaves the plain matcher in use.  With limits the
 * matcher runs one workgroup per switch group: a unicast switch's
 * out-neighbours, and a limited switch together with its out-neighbours,
 * form one group.  PCCL_EUNSUPPORTED (from pccl_workspace_bytes /
 * pccl_set_workspace) when a group has more than 768 in-links, 768
 * distinct sources of those links, 6144 in-links of those sources, a source
 * with more than 64 in-links, 64 limited or unicast switches, or more than
 * 1024 buffer places (capacities at or above the chunk count count as
 * unlimited).  With limited switches the workspace also holds a 4-byte
 * count per chunk for every limited switch plus one spare row per group
 * (16 MiB for the 512-NPU rail cluster's eight limited switches).  Buffers
 * can deadlock: then pccl_synthesize returns PCCL_EDEADLOCK.  PCCL_EINVAL
 * on a count mismatch.
 */
pccl_status pccl_set_switch_model(pccl_ctx *ctx, uint32_t n_switches, const uint32_t *buffer_chunks,
                                  const uint8_t *unicast);

/*
 * Device workspace needed by pccl_synthesize for at most `max_sends`
 * copy-schedule transfers (0 = the safe bound C * (D - 1), D = all devices).
 * The number of copy transfers equals the number of (device, chunk) pairs
 * that must receive the chunk: destinations plus relays.  The bound is an
 * argument because the send log, the output and the sort buffers (44 bytes
 * per transfer) scale with it: the safe bound of the 512-NPU All-to-All is
 * 136 M transfers (6 GB), its exact count 745,472 (33 MB).
 */
pccl_status pccl_workspace_bytes(pccl_ctx *ctx, uint64_t max_sends, size_t *out_bytes);

/*
 * Hands over the device workspace (caller-owned, 256-byte aligned, at least
 * the size pccl_workspace_bytes returned for `max_sends`) and the HIP stream
 * to run on (NULL = the default stream).  The library allocates no device
 * memory of its own (a context holds pinned host memory: the copies of the
 * inputs and of its small tables, and a 2 x 160-byte block for reading the
 * device's counters).  The workspace must not be used by the caller while a
 * synthesize call runs.  PCCL_ENOMEM if `bytes` is too small.
 */
pccl_status pccl_set_workspace(pccl_ctx *ctx, void *device_ptr, size_t bytes,
                               uint64_t max_sends, void *hip_stream);

/*
 * Runs the whole synthesis on the device and waits for it: the copy of the
 * inputs into the workspace (on the first call after pccl_set_collective or
 * pccl_set_workspace), conditions, shortest-path distances and relay devices
 * (Alg. 3 distances; the path-filtering step after Alg. 2), priority order
 * (Alg. 3), the event-stepped link-parallel matching (the BFS step of Alg. 2
 * applied to all free links at once; link exclusivity of Sec. 4.4 and 4.6;
 * chunk arrival times of Sec. 4.6; NextAvailableTime of Alg. 1), and the
 * canonical schedule (sorted by start time, then link id; reversed for
 * reduction ops).  Allocates nothing.
 * Outputs the number of sends and the collective time (latest transfer end).
 * The schedule stays in the workspace until the next synthesize call.
 * PCCL_ENOMEM if the collective needs more than max_sends transfers.
 */
pccl_status pccl_synthesize(pccl_ctx *ctx, uint64_t *n_sends, uint32_t *collective_time_ns);

/* Size of the library's static scratch: one device array per GPU the
 * library runs on, held until the process ends (pccl_synthesize_static). */
#define PCCL_STATIC_SCRATCH_BYTES (128ull << 20)

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation: the same
 * synthesis as pccl_set_workspace + pccl_synthesize, run in the library's
 * static scratch (PCCL_STATIC_SCRATCH_BYTES of device memory per GPU, a
 * file-scope array whose address pccl_create looks up once per device)
 * instead of a caller workspace.  The call allocates nothing and calls no
 * allocating routine.
 *   max_sends: bound on the copy transfers, as for pccl_workspace_bytes
 *     (0 = the safe bound C * (D - 1), which only small collectives fit).
 *   hip_stream: the stream to run on (NULL = the default stream).
 * PCCL_ENOMEM, with the sizes in pccl_last_error, when the collective's
 * workspace for max_sends exceeds PCCL_STATIC_SCRATCH_BYTES (the 512-NPU
 * All-to-All with its exact 745,472 transfers needs ~103 MiB and fits);
 * otherwise the statuses of pccl_synthesize.  The context's workspace is
 * then the scratch: pccl_get_schedule and the other readers copy from it
 * until a later call of this function on the same GPU, by any context,
 * reuses the scratch; they then return PCCL_ESTATE.  Every call on a GPU
 * shares that GPU's scratch: calls that overlap on one GPU (several threads,
 * or streams without ordering) race and must not be made.  The inputs are
 * copied into the scratch again unless this context, with the same
 * collective and max_sends, was the last to use it.
 */
pccl_status pccl_synthesize_static(pccl_ctx *ctx, uint64_t max_sends, void *hip_stream, uint64_t *n_sends,
                                   uint32_t *collective_time_ns);

/* Copies the schedule (canonical order) to `out`, host or device memory,
 * at most `capacity` entries.  PCCL_EINVAL if capacity is too small. */
pccl_status pccl_get_schedule(pccl_ctx *ctx, pccl_send *out, uint64_t capacity);

/*
 * The schedule in the paper's path form (Sec. 4.3, BFS pathfinding: a path
 * is an ordered list of (t, n) -- the chunk is sent from where it is to
 * device n at time t -- and a condition's result maps each destination to
 * its path).  Writes the path of `chunk` (caller's chunk id) from its
 * source to `device`: entry i is sent at t_start[i] (ns) to next_device[i];
 * the last entry is `device` itself, relays (switches, devices outside the
 * group) appear as intermediate entries.  *length receives the number of
 * hops; entries beyond `capacity` are not written (call again with a larger
 * buffer).  For reduction ops the path is the one of the dual copy schedule
 * (before reversal).  Output arrays are HOST memory.
 * PCCL_ESTATE without a schedule, PCCL_EINVAL for a chunk or device out of
 * range, a null output with capacity > 0, or a device that receives no
 * copy of the chunk (its source included).
 */
pccl_status pccl_get_path(pccl_ctx *ctx, uint32_t chunk, uint32_t device, uint32_t *t_start,
                          uint32_t *next_device, uint32_t capacity, uint32_t *length);

/*
 * The schedule as a program for GPUs that execute it (the translation of
 * synthesis results to MSCCL-style representations, Sec. 4.8): switches are
 * folded away, so each transfer runs directly from NPU to NPU over the
 * fabric (a chunk forwarded by a switch goes from the NPU that sent it into
 * the switch to each NPU the switch sends it to; a partial sum sent into a
 * switch goes to where the switch sends it on).  Rank r gets one thread
 * block per peer it sends to and one per peer it receives from (send blocks
 * by ascending peer first, then receive blocks); a block's steps are its
 * transfers in (start time, chunk) order.  Each transfer is a SEND step on
 * the sender and a RECV step (RECV_REDUCE for a reduction transfer) on the
 * receiver.  A SEND of chunk c on rank r waits for every receive of c on r
 * that ends before it starts (the chunk, or the partial sums of its
 * reduction subtree, must be there).
 * Steps are written ordered by (rank, tb, position in the block); `deps`
 * holds step indices.  Output arrays are HOST memory.  *n_steps / *n_deps
 * receive the sizes.  With steps and deps both NULL the call only sizes the
 * buffers; with a buffer smaller than needed nothing is written
 * (PCCL_EINVAL).  PCCL_ESTATE without a schedule.
 */
pccl_status pccl_export_program(pccl_ctx *ctx, pccl_step *steps, uint64_t step_capacity, uint32_t *deps,
                                uint64_t dep_capacity, uint64_t *n_steps, uint64_t *n_deps);

/*
 * Link usage of the schedule (the quantities behind the paper's link
 * utilization heat map and bandwidth-over-time figures, Sec. 6.4), computed
 * on the host from the last synthesize call's schedule (all of it: both
 * halves of an All-Reduce):
 *   busy_ns[L]: time link l carries transfers, the sum of T[l] over its
 *     sends (its busy fraction is busy_ns[l] / collective time);
 *   bin_busy_ns[n_bins]: the collective time cut into n_bins bins of
 *     *bin_ns = ceil(collective time / n_bins) ns; entry b is the link-time
 *     of all transfers inside bin b (utilization over time = bin_busy_ns[b]
 *     / (L * bin_ns)).
 * Output arrays are HOST memory; either may be NULL (n_bins is then
 * ignored).  PCCL_ESTATE without a schedule, PCCL_EINVAL for n_bins == 0
 * with bin_busy_ns given.
 */
pccl_status pccl_get_link_usage(pccl_ctx *ctx, uint64_t *busy_ns, uint32_t n_bins, uint64_t *bin_busy_ns,
                                uint32_t *bin_ns);

/*
 * Statistics of the last synthesize call:
 *   events  -- distinct event times visited by the event loop (time 0 plus
 *              every transfer end up to the last transfer start),
 *   rounds  -- (event, destination) pick rounds that made at least one pick,
 *   clashes -- picks that lost a (destination, chunk) clash,
 *   windows -- synchronous look-ahead windows the device loop ran (the
 *              device's own step count: events inside one window of the
 *              smallest link time need no grid-wide exchange, so this is
 *              what bounds the matching time, not `events`).
 * Any pointer may be NULL.
 */
pccl_status pccl_get_stats(pccl_ctx *ctx, uint64_t *events, uint64_t *rounds,
                           uint64_t *clashes, uint64_t *windows);

/*
 * Which matching kernel produced the last schedule: *kernel = 0 for the
 * event-stepped kernel with one wavefront per destination, 1 for the
 * switch-group kernel of the switch model (Sec. 4.7).  With a switch model
 * that has no binding buffer limit, the second runs only when two
 * out-neighbours of one unicast switch need the same chunk (checked on the
 * device after the setup); otherwise the no-multicast rule can never act and
 * the first gives the same schedule.  PCCL_ESTATE before a schedule exists.
 */
pccl_status pccl_get_matcher(pccl_ctx *ctx, uint32_t *kernel);

/*
 * Setup products of the last synthesize call, copied to host arrays (any may
 * be NULL): link_time_ns[L] = alpha + ceil(m / bw); chunk_src[C] (source NPU
 * or 0xFFFFFFFF when the chunk is unused); chunk_dist[C] (max shortest-path
 * distance in ns from the source to the destinations, 0 if none);
 * chunk_rank[C] (position in the priority order).
 */
pccl_status pccl_get_setup(pccl_ctx *ctx, uint32_t *link_time_ns, uint32_t *chunk_src,
                           uint64_t *chunk_dist, uint32_t *chunk_rank);

/*
 * Timing and work counters of the last synthesize call, measured with HIP
 * events recorded on the library's stream around its three stages: setup
 * (conditions to initial bitmaps, and the copy of the delivery count to the
 * host), matching (the persistent event-loop kernel) and output (canonical
 * sort and reversal, queued while the matching kernel runs).  scan_words counts the
 * word positions of the two rows the intersect passed (from a link's cursor
 * through the word holding its pick, or to the end of the row's own
 * ceil(chunks / 64) words when it found none), including the positions a
 * busy link's look-ahead passed; each position is one 64-bit word of each
 * row.  Any pointer may be NULL.
 */
pccl_status pccl_get_profile(pccl_ctx *ctx, double *setup_ms, double *match_ms, double *output_ms,
                             uint64_t *scan_words);

/* Message of the last failed call on this context ("" if none). */
const char *pccl_last_error(const pccl_ctx *ctx);

#ifdef __cplusplus
}
#endif
#endif /* PCCL_H */
