/*
 * pccl_oracle.c -- CPU oracle of the PCCL synthesis matcher.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg do.  It shares no code, header or table with the HIP
 * library: it is a plain, slow, single-threaded restatement of the method,
 * written so that every step can be checked against the paper by eye.
 *
 * What it computes (paper: "PCCL: Process Group-Aware Scalable and Generic
 * Collective Algorithm Synthesizer"):
 *   - conditions: one source and a destination set per chunk, derived from
 *     the NPU-centric pre/postconditions (Sec. 4.1 "Condition");
 *   - link transfer time alpha + m * beta with beta = 1 / bandwidth
 *     (Sec. 4.6, alpha-beta model), in whole nanoseconds rounded up;
 *   - per-condition distance = the maximum shortest-path distance from the
 *     source to its destinations, and the descending-distance processing
 *     order (Alg. 3, Sec. 4.4);
 *   - relay devices: shortest-path trees over the whole network pruned to the
 *     paths that reach the destinations, so devices outside the process group
 *     forward chunks (Sec. 4.3, the path-filtering step after Alg. 2);
 *   - an event-stepped, link-parallel greedy matching over the time-expanded
 *     network: a link may start a transfer when its source holds the chunk and
 *     its destination has not got it (the BFS step of Alg. 2), a link carries
 *     one chunk at a time for its whole alpha-beta duration (Sec. 4.4 link
 *     removal, and the overlapping-link removal of Sec. 4.6), a chunk may be
 *     forwarded once it has arrived (Sec. 4.6 "Chunk Arrival Time"), and time
 *     advances to the next moment a link becomes available (NextAvailableTime
 *     of Alg. 1);
 *   - reductions by time-reversing the dual non-reduction schedule, and
 *     All-Reduce as the reversed schedule followed by the forward one
 *     (Sec. 4.5);
 *   - optionally, explicit switch nodes (Sec. 4.7 "Modeling Switches"): a
 *     switch with a finite buffer accepts a new chunk only while fewer chunks
 *     than its capacity are buffered there, and a switch without multicast
 *     forwards one copy of a chunk at a time.
 * The readings taken where the paper is silent (tie-breaks, rounding, the
 * clash rule, relay needs) are listed in the repository's design notes; each
 * is restated at the step it governs below.
 *
 * Parity pins (tests/ check this file against them, never against the GPU):
 * ring All-Gather closed forms, complete-graph All-to-All, broadcast depth,
 * forced relay paths, the 2-level switch structure, hand-worked clash and
 * priority examples, schedule invariants, brute-force optimal makespans on
 * tiny inputs, Floyd-Warshall distances and SplitMix64 reference vectors.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <stdarg.h>

#define OR_OK 0
#define OR_EINVAL 1
#define OR_EUNREACHABLE 2
#define OR_ERANGE 3
#define OR_ENOMEM 4
#define OR_EUNSUPPORTED 7
#define OR_EDEADLOCK 8

#define OP_COPY 0
#define OP_REDUCE_REVERSED 1
#define OP_ALLREDUCE 2

#define NONE 0xFFFFFFFFu
#define INF64 0xFFFFFFFFFFFFFFFFull

typedef struct {
    uint32_t link, chunk, t_start, flags;
} or_send;

typedef struct {
    int status;
    char msg[256];
    /* setup products (user chunk order) */
    uint32_t n_links, n_chunks, n_devices;
    uint32_t *T;          /* [L] link time in ns */
    uint32_t *chunk_src;  /* [C] source NPU or NONE */
    uint64_t *chunk_dist; /* [C] max shortest-path distance to dests */
    uint32_t *rank;       /* [C] priority position of each chunk */
    uint64_t needs_total; /* initial number of needs bits */
    /* schedule */
    uint64_t n_sends;
    or_send *sends;
    uint32_t collective_time;
    /* statistics */
    uint64_t events, rounds, clashes, wasted, scan_words;
} or_result;

static int fail(or_result *r, int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(r->msg, sizeof r->msg, fmt, ap);
    va_end(ap);
    r->status = code;
    return code;
}

static int bit_get(const uint64_t *row, uint64_t c) { return (int)((row[c >> 6] >> (c & 63)) & 1u); }
static void bit_set(uint64_t *row, uint64_t c) { row[c >> 6] |= 1ull << (c & 63); }
static void bit_clr(uint64_t *row, uint64_t c) { row[c >> 6] &= ~(1ull << (c & 63)); }

/* SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): output number c+1 of the
 * generator started at state `seed`.  Used as the seeded tie-break key. */
static uint64_t splitmix64_output(uint64_t seed, uint64_t c)
{
    uint64_t z = seed + (c + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* chunk ordering: distance descending, then tie-break key ascending, then id */
static const uint64_t *g_dist;
static const uint64_t *g_key;
static int cmp_priority(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    if (g_dist[x] != g_dist[y]) return g_dist[x] > g_dist[y] ? -1 : 1;
    if (g_key[x] != g_key[y]) return g_key[x] < g_key[y] ? -1 : 1;
    return x < y ? -1 : (x > y);
}

static int cmp_send(const void *a, const void *b)
{
    const or_send *x = a, *y = b;
    if (x->t_start != y->t_start) return x->t_start < y->t_start ? -1 : 1;
    return x->link < y->link ? -1 : (x->link > y->link);
}

/* Plain O(D^2) Dijkstra from `s` over link times T (textbook form). */
static void dijkstra(uint32_t D, uint32_t s, const uint32_t *out_off, const uint32_t *out_link,
                     const uint32_t *ldst, const uint32_t *T, uint64_t *dist, char *done)
{
    for (uint32_t v = 0; v < D; v++) { dist[v] = INF64; done[v] = 0; }
    dist[s] = 0;
    for (;;) {
        uint32_t u = NONE;
        for (uint32_t v = 0; v < D; v++)
            if (!done[v] && dist[v] != INF64 && (u == NONE || dist[v] < dist[u])) u = v;
        if (u == NONE) break;
        done[u] = 1;
        for (uint32_t k = out_off[u]; k < out_off[u + 1]; k++) {
            uint32_t l = out_link[k], v = ldst[l];
            if (dist[u] + T[l] < dist[v]) dist[v] = dist[u] + T[l];
        }
    }
}

/*
 * mode bit 0: skip the rescan of a free link whose candidate set was found
 * empty and whose source has received nothing since (result-identical: the
 * destination's needs only shrink, so the candidate set of such a link stays
 * empty; the one other way a candidate reappears is a unicast switch source
 * finishing a copy, which wakes that switch's out-links too).  Without it
 * every free link rescans at every event, as the event loop is stated.
 */
/*
 * Switch model (Sec. 4.7), both arrays indexed by switch (device N + i), NULL
 * for none:
 *   sw_buffer[i]  0 = unlimited; else the most chunks switch i buffers at
 *                 once.  A chunk counts as buffered at switch w from the start
 *                 of its transfer into w until no out-neighbour of w still
 *                 needs it; a transfer into w may start only while fewer than
 *                 sw_buffer chunks are buffered there (visiting w would
 *                 otherwise exceed its buffer).  Several transfers into w that
 *                 win their clashes in the same round take the free places in
 *                 (link time, link id) order; the others stay in the round loop.
 *   sw_unicast[i] 1 = no multicast: switch i never has two copies of one chunk
 *                 in flight on its out-links (it visits its next neighbours
 *                 one by one).  A free out-link of i skips chunks i is
 *                 sending; out-links of i that pick the same chunk in one round
 *                 clash, after the destination clash, with the same rule
 *                 (fastest link, then lowest id).
 */
int pccl_oracle_run(uint32_t n_npus, uint32_t n_switches, uint32_t n_links,
                    const uint32_t *lsrc, const uint32_t *ldst, const uint32_t *alpha,
                    const uint32_t *bw, uint32_t C, uint64_t m, const uint64_t *pre,
                    const uint64_t *post, const uint64_t *group_masks, uint32_t n_groups,
                    const uint16_t *chunk_group, int op, uint64_t tie_seed, int mode,
                    const uint32_t *sw_buffer, const uint8_t *sw_unicast, void **handle)
{
    or_result *r = calloc(1, sizeof *r);
    *handle = r;
    if (!r) return OR_ENOMEM;
    const uint32_t N = n_npus, D = n_npus + n_switches, L = n_links;
    const uint64_t W = ((uint64_t)C + 63) / 64;      /* words per chunk row */
    const uint64_t WN = ((uint64_t)N + 63) / 64;     /* words per group mask */
    r->n_links = L;
    r->n_chunks = C;
    r->n_devices = D;

    /* ---------------- input checks ---------------- */
    if (N == 0) return fail(r, OR_EINVAL, "no NPUs");
    if (m == 0) return fail(r, OR_EINVAL, "chunk size 0");
    if (n_groups == 0) return fail(r, OR_EINVAL, "no process group");
    if (n_groups > 1 && !chunk_group) return fail(r, OR_EINVAL, "several groups need chunk_group");
    for (uint32_t l = 0; l < L; l++) {
        if (lsrc[l] >= D || ldst[l] >= D) return fail(r, OR_EINVAL, "link %u endpoint out of range", l);
        if (lsrc[l] == ldst[l]) return fail(r, OR_EINVAL, "link %u is a self loop", l);
        if (bw[l] == 0) return fail(r, OR_EINVAL, "link %u has zero bandwidth", l);
        for (uint32_t k = 0; k < l; k++)
            if (lsrc[k] == lsrc[l] && ldst[k] == ldst[l])
                return fail(r, OR_EINVAL, "links %u and %u are duplicates", k, l);
    }
    for (uint32_t g = 0; g < n_groups; g++)
        for (uint32_t v = N; v < WN * 64; v++)
            if (bit_get(group_masks + g * WN, v)) return fail(r, OR_EINVAL, "group %u names a non-NPU", g);
    if (chunk_group)
        for (uint32_t c = 0; c < C; c++)
            if (chunk_group[c] >= n_groups) return fail(r, OR_EINVAL, "chunk %u has bad group", c);

    /* link time: alpha + ceil(m / bandwidth); 1 GB/s is 1 byte per ns */
    r->T = malloc(sizeof(uint32_t) * (L ? L : 1));
    for (uint32_t l = 0; l < L; l++) {
        uint64_t beta_part = m / bw[l] + (m % bw[l] != 0);
        uint64_t t = (uint64_t)alpha[l] + beta_part;
        if (beta_part > 0xFFFFFFFFull || t > 0xFFFFFFFFull)
            return fail(r, OR_ERANGE, "link %u time does not fit in 32 bits", l);
        r->T[l] = (uint32_t)t;
    }
    const uint32_t *T = r->T;

    if (op == OP_REDUCE_REVERSED || op == OP_ALLREDUCE) {
        for (uint32_t l = 0; l < L; l++) {
            uint32_t rv = NONE;
            for (uint32_t k = 0; k < L; k++)
                if (lsrc[k] == ldst[l] && ldst[k] == lsrc[l]) rv = k;
            if (rv == NONE || T[rv] != T[l])
                return fail(r, OR_EUNSUPPORTED, "link %u has no reverse link of equal time", l);
        }
    } else if (op != OP_COPY) {
        return fail(r, OR_EINVAL, "unknown op %d", op);
    }

    /* conditions: the unique precondition holder and the destinations */
    r->chunk_src = malloc(sizeof(uint32_t) * (C ? C : 1));
    r->chunk_dist = calloc(C ? C : 1, sizeof(uint64_t));
    r->rank = malloc(sizeof(uint32_t) * (C ? C : 1));
    for (uint64_t k = (uint64_t)C; k < W * 64; k++)
        for (uint32_t v = 0; v < N; v++)
            if (bit_get(pre + v * W, k) || bit_get(post + v * W, k))
                return fail(r, OR_EINVAL, "bit set beyond the last chunk");
    for (uint32_t c = 0; c < C; c++) {
        uint32_t g = chunk_group ? chunk_group[c] : 0;
        const uint64_t *gm = group_masks + (uint64_t)g * WN;
        uint32_t holders = 0, src = NONE, posts = 0;
        for (uint32_t v = 0; v < N; v++) {
            int p = bit_get(pre + v * W, c), q = bit_get(post + v * W, c);
            if ((p || q) && !bit_get(gm, v))
                return fail(r, OR_EINVAL, "chunk %u has a pre/post bit on non-member %u", c, v);
            if (p) { holders++; src = v; }
            if (q) posts++;
        }
        if (holders > 1) return fail(r, OR_EINVAL, "chunk %u has %u holders", c, holders);
        if (holders == 0 && posts > 0) return fail(r, OR_EINVAL, "chunk %u is needed but held by nobody", c);
        r->chunk_src[c] = src;
    }

    /* out-adjacency for Dijkstra */
    uint32_t *out_off = calloc(D + 1, sizeof(uint32_t));
    uint32_t *out_link = malloc(sizeof(uint32_t) * (L ? L : 1));
    for (uint32_t l = 0; l < L; l++) out_off[lsrc[l] + 1]++;
    for (uint32_t v = 0; v < D; v++) out_off[v + 1] += out_off[v];
    {
        uint32_t *fill = calloc(D, sizeof(uint32_t));
        for (uint32_t l = 0; l < L; l++) out_link[out_off[lsrc[l]] + fill[lsrc[l]]++] = l;
        free(fill);
    }

    /* in-links per destination: tight predecessors and clash groups */
    uint32_t *in_off = calloc(D + 1, sizeof(uint32_t));
    uint32_t *in_link = malloc(sizeof(uint32_t) * (L ? L : 1));
    for (uint32_t l = 0; l < L; l++) in_off[ldst[l] + 1]++;
    for (uint32_t v = 0; v < D; v++) in_off[v + 1] += in_off[v];
    {
        uint32_t *fill = calloc(D, sizeof(uint32_t));
        for (uint32_t l = 0; l < L; l++) in_link[in_off[ldst[l]] + fill[ldst[l]]++] = l;
        free(fill);
    }

    /* shortest-path distance and parent (smallest-id tight predecessor) per source */
    uint64_t *dist = malloc(sizeof(uint64_t) * (uint64_t)N * D);
    uint32_t *parent = malloc(sizeof(uint32_t) * (uint64_t)N * D);
    char *have = calloc(N, 1), *done = malloc(D);
    for (uint32_t c = 0; c < C; c++)
        if (r->chunk_src[c] != NONE) have[r->chunk_src[c]] = 1;
    for (uint32_t s = 0; s < N; s++) {
        if (!have[s]) continue;
        uint64_t *ds = dist + (uint64_t)s * D;
        uint32_t *ps = parent + (uint64_t)s * D;
        dijkstra(D, s, out_off, out_link, ldst, T, ds, done);
        for (uint32_t v = 0; v < D; v++) {
            ps[v] = NONE;
            if (v == s || ds[v] == INF64) continue;
            for (uint32_t k = in_off[v]; k < in_off[v + 1]; k++) {
                uint32_t l = in_link[k];
                if (ds[lsrc[l]] != INF64 && ds[lsrc[l]] + T[l] == ds[v] && (ps[v] == NONE || lsrc[l] < ps[v]))
                    ps[v] = lsrc[l];
            }
        }
    }
    free(done);

    /* condition distance: max over destinations (destinations = post and not pre) */
    for (uint32_t c = 0; c < C; c++) {
        uint32_t s = r->chunk_src[c];
        if (s == NONE) continue;
        for (uint32_t v = 0; v < N; v++) {
            if (!bit_get(post + v * W, c) || bit_get(pre + v * W, c)) continue;
            uint64_t dv = dist[(uint64_t)s * D + v];
            if (dv == INF64) return fail(r, OR_EUNREACHABLE, "chunk %u: NPU %u unreachable from %u", c, v, s);
            if (dv >= 0xFFFFFFFFull) return fail(r, OR_ERANGE, "chunk %u: distance does not fit in 32 bits", c);
            if (dv > r->chunk_dist[c]) r->chunk_dist[c] = dv;
        }
    }

    /* priority: distance descending, seeded SplitMix64 key ascending, chunk id */
    uint64_t *key = malloc(sizeof(uint64_t) * (C ? C : 1));
    uint32_t *order = malloc(sizeof(uint32_t) * (C ? C : 1));
    for (uint32_t c = 0; c < C; c++) { key[c] = splitmix64_output(tie_seed, c); order[c] = c; }
    g_dist = r->chunk_dist;
    g_key = key;
    qsort(order, C, sizeof(uint32_t), cmp_priority);
    for (uint32_t k = 0; k < C; k++) r->rank[order[k]] = k;

    /* initial state over rank-ordered columns: holds = precondition,
     * needs = destinations plus the relays on the pruned shortest-path tree */
    uint64_t *holds = calloc((uint64_t)D * W + 1, sizeof(uint64_t));
    uint64_t *needs = calloc((uint64_t)D * W + 1, sizeof(uint64_t));
    for (uint32_t c = 0; c < C; c++) {
        uint32_t s = r->chunk_src[c], q = r->rank[c];
        if (s == NONE) continue;
        bit_set(holds + (uint64_t)s * W, q);
        for (uint32_t v = 0; v < N; v++) {
            if (!bit_get(post + v * W, c) || bit_get(pre + v * W, c)) continue;
            bit_set(needs + (uint64_t)v * W, q);
            for (uint32_t u = parent[(uint64_t)s * D + v]; u != s; u = parent[(uint64_t)s * D + u])
                bit_set(needs + (uint64_t)u * W, q);
        }
    }
    free(dist);
    free(parent);
    free(have);
    uint64_t needs_remaining = 0;
    for (uint64_t k = 0; k < (uint64_t)D * W; k++) needs_remaining += (uint64_t)__builtin_popcountll(needs[k]);
    r->needs_total = needs_remaining;

    /* ---------------- event loop ---------------- */
    uint32_t *busy_until = calloc(L ? L : 1, sizeof(uint32_t));
    uint32_t *inflight = malloc(sizeof(uint32_t) * (L ? L : 1));
    uint32_t *pick = malloc(sizeof(uint32_t) * (L ? L : 1));
    char *active = calloc(L ? L : 1, 1), *win = calloc(L ? L : 1, 1);
    char *win2 = calloc(L ? L : 1, 1), *win3 = calloc(L ? L : 1, 1);
    uint32_t *occ = calloc(D, sizeof(uint32_t));  /* chunks buffered at each limited switch */
#define SW_BUF(v) ((sw_buffer && (v) >= N) ? sw_buffer[(v) - N] : 0u)
#define SW_UNI(v) ((sw_unicast && (v) >= N) ? sw_unicast[(v) - N] != 0 : 0)
    char *idle = calloc(L ? L : 1, 1);      /* mode bit 0 only */
    char *dst_picked = calloc(D, 1);
    for (uint32_t l = 0; l < L; l++) inflight[l] = NONE;
    uint64_t cap = needs_remaining ? needs_remaining : 1, ns = 0;
    or_send *log = malloc(sizeof(or_send) * cap);
    uint32_t t = 0;
    int status = OR_OK;

    for (;;) {
        r->events++;
        /* arrivals: a link whose transfer ends now delivers and becomes free */
        for (uint32_t l = 0; l < L; l++) {
            if (inflight[l] != NONE && busy_until[l] == t) {
                bit_set(holds + (uint64_t)ldst[l] * W, inflight[l]);
                inflight[l] = NONE;
                if (mode & 1) {
                    for (uint32_t k = out_off[ldst[l]]; k < out_off[ldst[l] + 1]; k++) idle[out_link[k]] = 0;
                    /* a unicast switch that finished a copy may send that chunk again */
                    if (SW_UNI(lsrc[l]))
                        for (uint32_t k = out_off[lsrc[l]]; k < out_off[lsrc[l] + 1]; k++) idle[out_link[k]] = 0;
                }
            }
        }
        /* rounds: every free link picks; clashes on (destination, chunk) are
         * won by the fastest link, then the lowest link id; losers pick again */
        uint32_t n_active = 0;
        for (uint32_t l = 0; l < L; l++) {
            active[l] = (inflight[l] == NONE) && !((mode & 1) && idle[l]);
            n_active += active[l];
        }
        while (n_active > 0) {
            /* buffered chunks of each limited switch w: present at w or in
             * flight into it, and still needed by an out-neighbour of w */
            for (uint32_t w = N; w < D; w++) {
                if (!SW_BUF(w)) continue;
                occ[w] = 0;
                for (uint32_t q = 0; q < C; q++) {
                    int present = bit_get(holds + (uint64_t)w * W, q);
                    for (uint32_t k = in_off[w]; k < in_off[w + 1] && !present; k++)
                        present = inflight[in_link[k]] == q;
                    if (!present) continue;
                    int wanted = 0;
                    for (uint32_t k = out_off[w]; k < out_off[w + 1] && !wanted; k++)
                        wanted = bit_get(needs + (uint64_t)ldst[out_link[k]] * W, q);
                    occ[w] += (uint32_t)wanted;
                }
            }
            int any = 0;
            for (uint32_t l = 0; l < L; l++) {
                if (!active[l]) continue;
                const uint32_t s = lsrc[l], d = ldst[l];
                const uint64_t *h = holds + (uint64_t)s * W, *nd = needs + (uint64_t)d * W;
                pick[l] = NONE;
                /* a full switch buffer admits nothing: the link stays in the
                 * round loop (a later round may free a place) */
                if (SW_BUF(d) && occ[d] >= SW_BUF(d)) continue;
                for (uint64_t k = 0; k < W && pick[l] == NONE; k++) {
                    r->scan_words++;
                    uint64_t x = h[k] & nd[k];
                    for (; x; x &= x - 1) {
                        const uint32_t c = (uint32_t)(k * 64 + (uint64_t)__builtin_ctzll(x));
                        int sending = 0;  /* a unicast switch already sends c */
                        if (SW_UNI(s))
                            for (uint32_t o = out_off[s]; o < out_off[s + 1] && !sending; o++)
                                sending = inflight[out_link[o]] == c;
                        if (!sending) { pick[l] = c; break; }
                    }
                }
                if (pick[l] == NONE) {
                    active[l] = 0;
                    n_active--;
                    if (mode & 1) idle[l] = 1;
                } else {
                    any = 1;
                }
            }
            if (!any) break;
            /* clash on (destination, chunk) */
            for (uint32_t l = 0; l < L; l++) {
                if (!active[l] || pick[l] == NONE) continue;
                win[l] = 1;
                uint32_t d = ldst[l];
                for (uint32_t k = in_off[d]; k < in_off[d + 1]; k++) {
                    uint32_t o = in_link[k];
                    if (o == l || !active[o] || pick[o] != pick[l]) continue;
                    if (T[o] < T[l] || (T[o] == T[l] && o < l)) win[l] = 0;
                }
                if (!dst_picked[d]) { dst_picked[d] = 1; r->rounds++; }
            }
            /* clash on (unicast switch, chunk) among the destination winners */
            for (uint32_t l = 0; l < L; l++) {
                if (!active[l] || pick[l] == NONE) continue;
                win2[l] = win[l];
                const uint32_t s = lsrc[l];
                if (!win[l] || !SW_UNI(s)) continue;
                for (uint32_t k = out_off[s]; k < out_off[s + 1]; k++) {
                    uint32_t o = out_link[k];
                    if (o == l || !active[o] || pick[o] == NONE || !win[o] || pick[o] != pick[l]) continue;
                    if (T[o] < T[l] || (T[o] == T[l] && o < l)) win2[l] = 0;
                }
            }
            /* free places of a limited switch buffer, in (link time, link id) order */
            for (uint32_t l = 0; l < L; l++) {
                if (!active[l] || pick[l] == NONE) continue;
                win3[l] = win2[l];
                const uint32_t d = ldst[l];
                if (!win2[l] || !SW_BUF(d)) continue;
                uint32_t ahead = 0;
                for (uint32_t k = in_off[d]; k < in_off[d + 1]; k++) {
                    uint32_t o = in_link[k];
                    if (o == l || !active[o] || pick[o] == NONE || !win2[o]) continue;
                    if (T[o] < T[l] || (T[o] == T[l] && o < l)) ahead++;
                }
                if (ahead >= SW_BUF(d) - occ[d]) win3[l] = 0;
            }
            for (uint32_t l = 0; l < L; l++) {
                if (!active[l] || pick[l] == NONE) continue;
                dst_picked[ldst[l]] = 0;
                if (!win3[l]) { r->clashes++; continue; }
                uint64_t end = (uint64_t)t + T[l];
                if (end > 0xFFFFFFFFull) { status = fail(r, OR_ERANGE, "time does not fit in 32 bits"); goto done; }
                bit_clr(needs + (uint64_t)ldst[l] * W, pick[l]);
                inflight[l] = pick[l];
                busy_until[l] = (uint32_t)end;
                log[ns].link = l;
                log[ns].chunk = pick[l];
                log[ns].t_start = t;
                log[ns].flags = 0;
                ns++;
                needs_remaining--;
                active[l] = 0;
                n_active--;
            }
        }
        if (needs_remaining == 0) break;
        /* NextAvailableTime: advance to the earliest end of a transfer */
        uint32_t tn = NONE;
        int inflight_any = 0;
        for (uint32_t l = 0; l < L; l++)
            if (inflight[l] != NONE) {
                inflight_any = 1;
                if (busy_until[l] < tn) tn = busy_until[l];
            }
        if (!inflight_any) { status = fail(r, OR_EDEADLOCK, "needs remain but nothing is in flight"); goto done; }
        t = tn;
    }

    /* wasted relay deliveries: received by a non-destination that never forwards it */
    {
        uint64_t *fwd = calloc((uint64_t)D * W + 1, sizeof(uint64_t));
        for (uint64_t i = 0; i < ns; i++) bit_set(fwd + (uint64_t)lsrc[log[i].link] * W, log[i].chunk);
        for (uint64_t i = 0; i < ns; i++) {
            uint32_t v = ldst[log[i].link], c = order[log[i].chunk];
            int is_dest = v < N && bit_get(post + (uint64_t)v * W, c) && !bit_get(pre + (uint64_t)v * W, c);
            if (!is_dest && !bit_get(fwd + (uint64_t)v * W, log[i].chunk)) r->wasted++;
        }
        free(fwd);
    }

    /* output: caller's chunk ids, canonical (t_start, link) order */
    {
        uint32_t cstar = 0;
        for (uint64_t i = 0; i < ns; i++) {
            uint32_t e = log[i].t_start + T[log[i].link];
            if (e > cstar) cstar = e;
            log[i].chunk = order[log[i].chunk];
        }
        if (op == OP_COPY) {
            r->sends = log;
            r->n_sends = ns;
            r->collective_time = cstar;
            log = NULL;
        } else {
            uint64_t total = op == OP_ALLREDUCE ? 2 * ns : ns;
            if (op == OP_ALLREDUCE && 2ull * cstar > 0xFFFFFFFFull) {
                status = fail(r, OR_ERANGE, "all-reduce time does not fit in 32 bits");
                goto done;
            }
            or_send *out = malloc(sizeof(or_send) * (total ? total : 1));
            for (uint64_t i = 0; i < ns; i++) {
                uint32_t l = log[i].link, rv = NONE;
                for (uint32_t k = 0; k < L; k++)
                    if (lsrc[k] == ldst[l] && ldst[k] == lsrc[l]) rv = k;
                out[i].link = rv;
                out[i].chunk = log[i].chunk;
                out[i].t_start = cstar - log[i].t_start - T[l];
                out[i].flags = 1;
                if (op == OP_ALLREDUCE) {
                    out[ns + i] = log[i];
                    out[ns + i].t_start += cstar;
                }
            }
            r->sends = out;
            r->n_sends = total;
            r->collective_time = op == OP_ALLREDUCE ? 2 * cstar : cstar;
        }
        qsort(r->sends, r->n_sends, sizeof(or_send), cmp_send);
    }

done:
    free(log);
    free(holds);
    free(needs);
    free(in_off);
    free(in_link);
    free(out_off);
    free(out_link);
    free(busy_until);
    free(inflight);
    free(pick);
    free(active);
    free(win);
    free(win2);
    free(win3);
    free(occ);
    free(idle);
    free(dst_picked);
    free(key);
    free(order);
    r->status = status;
    return status;
}

int pccl_oracle_status(void *h) { return ((or_result *)h)->status; }
const char *pccl_oracle_message(void *h) { return ((or_result *)h)->msg; }
uint64_t pccl_oracle_n_sends(void *h) { return ((or_result *)h)->n_sends; }
uint32_t pccl_oracle_collective_time(void *h) { return ((or_result *)h)->collective_time; }

void pccl_oracle_sends(void *h, uint32_t *out4)
{
    or_result *r = h;
    for (uint64_t i = 0; i < r->n_sends; i++) {
        out4[4 * i + 0] = r->sends[i].link;
        out4[4 * i + 1] = r->sends[i].chunk;
        out4[4 * i + 2] = r->sends[i].t_start;
        out4[4 * i + 3] = r->sends[i].flags;
    }
}

/* events, rounds, clashes, wasted relay sends, scanned words, initial needs */
void pccl_oracle_stats(void *h, uint64_t *out6)
{
    or_result *r = h;
    out6[0] = r->events;
    out6[1] = r->rounds;
    out6[2] = r->clashes;
    out6[3] = r->wasted;
    out6[4] = r->scan_words;
    out6[5] = r->needs_total;
}

/* setup products, valid when setup got that far */
void pccl_oracle_setup(void *h, uint32_t *T, uint32_t *chunk_src, uint64_t *chunk_dist, uint32_t *rank)
{
    or_result *r = h;
    if (T && r->T) memcpy(T, r->T, sizeof(uint32_t) * r->n_links);
    if (chunk_src && r->chunk_src) memcpy(chunk_src, r->chunk_src, sizeof(uint32_t) * r->n_chunks);
    if (chunk_dist && r->chunk_dist) memcpy(chunk_dist, r->chunk_dist, sizeof(uint64_t) * r->n_chunks);
    if (rank && r->rank) memcpy(rank, r->rank, sizeof(uint32_t) * r->n_chunks);
}

uint64_t pccl_oracle_splitmix64(uint64_t seed, uint64_t c) { return splitmix64_output(seed, c); }

void pccl_oracle_free(void *h)
{
    or_result *r = h;
    if (!r) return;
    free(r->T);
    free(r->chunk_src);
    free(r->chunk_dist);
    free(r->rank);
    free(r->sends);
    free(r);
}
