// Condition-sequential synthesis taken literally: the breadth-first path
// search over the time-expanded network (TEN) of Alg. 2, run once per
// condition in the order of Alg. 3, with the interval links of Sec. 4.6.
//
// TEST INFRASTRUCTURE ONLY.  This is not what the GPU library computes (that
// is the link-parallel event loop, in pccl_oracle.c); it is the paper's own
// sequential procedure, kept to compare schedule quality.  Readings:
//  - the search advances time once per level, over a snapshot of the visited
//    set, so a chunk moves at most one hop per level; the next-time and
//    availability helpers of Alg. 1 return the time found and ask for the
//    next devices;
//  - heterogeneous links: a device sends only once the chunk has arrived; a
//    link s->d is present at time t when no transfer already placed on it
//    overlaps [t, t + T); time moves from one level to the next event (an
//    arrival, or the end of a busy interval on a link out of a reached
//    device), which visits exactly the levels where anything can change;
//  - within a level, reached devices in the order they were reached, and
//    each device's out-links by ascending destination id (then link id);
//  - after the search only the transfers on the paths to the condition's
//    destinations are kept, and they occupy their links;
//  - conditions in the order of Alg. 3: longest condition distance first,
//    ties by the seeded hash and the chunk id (given by the caller).
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define NONE 0xFFFFFFFFu

typedef struct {
    uint64_t s, e;  // busy over [s, e)
} ival;

typedef struct {
    ival *v;
    uint32_t n, cap;
} ivals;

// first interval with e > t (intervals are disjoint and sorted)
static uint32_t first_after(const ivals *iv, uint64_t t)
{
    uint32_t lo = 0, hi = iv->n;
    while (lo < hi) {
        const uint32_t mid = (lo + hi) / 2;
        if (iv->v[mid].e > t) hi = mid;
        else lo = mid + 1;
    }
    return lo;
}

static int is_free(const ivals *iv, uint64_t t, uint64_t T)
{
    const uint32_t i = first_after(iv, t);
    return i == iv->n || iv->v[i].s >= t + T;
}

// the earliest t' >= t with [t', t' + T) free
static uint64_t earliest_free(const ivals *iv, uint64_t t, uint64_t T)
{
    for (uint32_t i = first_after(iv, t); i < iv->n; i++) {
        if (iv->v[i].s >= t + T) return t;
        if (iv->v[i].e > t) t = iv->v[i].e;
    }
    return t;
}

static int occupy(ivals *iv, uint64_t s, uint64_t e)
{
    if (iv->n == iv->cap) {
        const uint32_t cap = iv->cap ? 2 * iv->cap : 8;
        ival *v = (ival *)realloc(iv->v, sizeof(ival) * cap);
        if (!v) return -1;
        iv->v = v;
        iv->cap = cap;
    }
    uint32_t i = first_after(iv, s);
    memmove(iv->v + i + 1, iv->v + i, sizeof(ival) * (iv->n - i));
    iv->v[i].s = s;
    iv->v[i].e = e;
    iv->n++;
    return 0;
}

typedef struct {
    uint32_t link, chunk;
    uint64_t t;
} alg3_send;

// Returns 0 on success, 2 when a destination cannot be reached, 4 on
// allocation failure, 8 when the search stalls.  `order` lists the
// conditions (chunk ids) in synthesis order; dest_off/dest_list give each
// chunk's destinations (CSR by chunk id).  *out receives malloc'ed sends in
// placement order (free with alg3_free).
int alg3_run(uint32_t D, uint32_t L, const uint32_t *lsrc, const uint32_t *ldst, const uint32_t *T,
             uint32_t n_cond, const uint32_t *order, const uint32_t *csrc, const uint64_t *dest_off,
             const uint32_t *dest_list, alg3_send **out, uint64_t *n_out, uint64_t *coll_time)
{
    int status = 4;
    *out = NULL;
    *n_out = 0;
    *coll_time = 0;
    // out-links by source, by ascending destination then link id
    uint32_t *ooff = (uint32_t *)calloc(D + 1, 4), *olink = (uint32_t *)malloc(4 * (L ? L : 1));
    ivals *busy = (ivals *)calloc(L ? L : 1, sizeof(ivals));
    uint64_t *arr = (uint64_t *)malloc(8 * (D ? D : 1));
    uint32_t *reached = (uint32_t *)malloc(4 * (D ? D : 1)), *plink = (uint32_t *)malloc(4 * (D ? D : 1));
    uint64_t *pt = (uint64_t *)malloc(8 * (D ? D : 1));
    char *used = (char *)calloc(D ? D : 1, 1);
    uint64_t cap = 1024, n = 0;
    alg3_send *sends = (alg3_send *)malloc(sizeof(alg3_send) * cap);
    if (!ooff || !olink || !busy || !arr || !reached || !plink || !pt || !used || !sends) goto done;
    for (uint32_t l = 0; l < L; l++) ooff[lsrc[l] + 1]++;
    for (uint32_t v = 0; v < D; v++) ooff[v + 1] += ooff[v];
    {
        uint32_t *fill = (uint32_t *)calloc(D ? D : 1, 4);
        if (!fill) goto done;
        for (uint32_t l = 0; l < L; l++) olink[ooff[lsrc[l]] + fill[lsrc[l]]++] = l;
        free(fill);
    }
    for (uint32_t v = 0; v < D; v++)  // insertion sort by (destination, link id)
        for (uint32_t i = ooff[v] + 1; i < ooff[v + 1]; i++) {
            const uint32_t x = olink[i];
            uint32_t j = i;
            while (j > ooff[v] && (ldst[olink[j - 1]] > ldst[x] || (ldst[olink[j - 1]] == ldst[x] && olink[j - 1] > x))) {
                olink[j] = olink[j - 1];
                j--;
            }
            olink[j] = x;
        }
    for (uint32_t k = 0; k < n_cond; k++) {
        const uint32_t c = order[k], src = csrc[c];
        const uint64_t d0 = dest_off[c], d1 = dest_off[c + 1];
        if (d0 == d1) continue;
        for (uint32_t v = 0; v < D; v++) arr[v] = UINT64_MAX;
        arr[src] = 0;
        uint32_t nr = 0;
        reached[nr++] = src;
        // first time the source has a link present (Alg. 1)
        uint64_t t = UINT64_MAX;
        for (uint32_t i = ooff[src]; i < ooff[src + 1]; i++) {
            const uint32_t l = olink[i];
            const uint64_t e = earliest_free(&busy[l], 0, T[l]);
            if (e < t) t = e;
        }
        if (t == UINT64_MAX) {
            status = 2;
            goto done;
        }
        uint64_t missing = 0;
        for (uint64_t q = d0; q < d1; q++) missing += dest_list[q] != src;
        while (missing) {
            const uint32_t level = nr;  // snapshot of the reached set
            for (uint32_t r = 0; r < level; r++) {
                const uint32_t cur = reached[r];
                if (arr[cur] > t) continue;  // the chunk is not there yet
                for (uint32_t i = ooff[cur]; i < ooff[cur + 1]; i++) {
                    const uint32_t l = olink[i], nx = ldst[l];
                    if (arr[nx] != UINT64_MAX || !is_free(&busy[l], t, T[l])) continue;
                    arr[nx] = t + T[l];
                    plink[nx] = l;
                    pt[nx] = t;
                    reached[nr++] = nx;
                    for (uint64_t q = d0; q < d1; q++)
                        if (dest_list[q] == nx) missing--;
                }
            }
            if (!missing) break;
            // the next level where anything can change
            uint64_t tn = UINT64_MAX;
            for (uint32_t r = 0; r < nr; r++) {
                const uint32_t v = reached[r];
                if (arr[v] > t) {
                    if (arr[v] < tn) tn = arr[v];
                    continue;
                }
                for (uint32_t i = ooff[v]; i < ooff[v + 1]; i++) {
                    const uint32_t l = olink[i];
                    if (arr[ldst[l]] != UINT64_MAX) continue;
                    const uint64_t e = earliest_free(&busy[l], t + 1, T[l]);
                    if (e < tn) tn = e;
                }
            }
            if (tn == UINT64_MAX) {
                status = 8;
                goto done;
            }
            t = tn;
        }
        // keep the paths to the destinations; they occupy their links
        for (uint64_t q = d0; q < d1; q++) {
            uint32_t v = dest_list[q];
            while (v != src && !used[v]) {
                used[v] = 1;
                const uint32_t l = plink[v];
                if (n == cap) {
                    cap *= 2;
                    alg3_send *s2 = (alg3_send *)realloc(sends, sizeof(alg3_send) * cap);
                    if (!s2) goto done;
                    sends = s2;
                }
                sends[n].link = l;
                sends[n].chunk = c;
                sends[n].t = pt[v];
                n++;
                if (occupy(&busy[l], pt[v], pt[v] + T[l])) goto done;
                if (pt[v] + T[l] > *coll_time) *coll_time = pt[v] + T[l];
                v = lsrc[l];
            }
        }
        for (uint32_t r = 0; r < nr; r++) used[reached[r]] = 0;
    }
    status = 0;
done:
    if (busy)
        for (uint32_t l = 0; l < L; l++) free(busy[l].v);
    free(busy);
    free(ooff);
    free(olink);
    free(arr);
    free(reached);
    free(plink);
    free(pt);
    free(used);
    if (status == 0) {
        *out = sends;
        *n_out = n;
    } else {
        free(sends);
    }
    return status;
}

void alg3_free(alg3_send *p) { free(p); }
