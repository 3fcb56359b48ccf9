// C ABI of the synthesis matcher: argument checks, the workspace layout,
// staging of the small topology arrays and the launch sequence.  All
// per-chunk and per-send work runs in the kernels of pccl_setup.hip,
// pccl_match.hip and pccl_sort.hip.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <exception>
#include <mutex>
#include <numeric>
#include <string>
#include <unordered_map>
#include <vector>

#include "pccl.h"
#include "pccl_internal.h"

using namespace pccl;

// The library's static scratch, for pccl_synthesize_static: a file-scope
// device array, one copy per GPU, held until the process ends.  Each device
// reports its copy's address once (hipGetSymbolAddress with that device
// current, from pccl_create); host code uses only those addresses, never
// the array's name.
static __device__ __align__(256) unsigned char scratch[PCCL_STATIC_SCRATCH_BYTES];

struct pccl_ctx {
    int device = 0;
    uint64_t seed = 0;
    std::string err;
    bool have_topo = false, have_coll = false, have_ws = false, uploaded = false, have_result = false;
    // topology
    uint32_t N = 0, S = 0, D = 0, L = 0;
    std::vector<uint32_t> src, dst, alpha, bw;
    std::vector<uint32_t> in_off, slot_link, slot_src, slot_cum, dest_pairs, rev;
    std::vector<uint32_t> wave_dest;  // destination of (pass, wave) in the matching kernel
    std::vector<uint32_t> wave_part;  // its part when the destination is split over a workgroup's waves
    std::vector<uint32_t> split;      // split destinations, each taking one workgroup (heaviest first)
    std::vector<std::vector<uint32_t>> split_cuts;  // their parts: first in-link of each part, then the in-degree
    bool resident = true;             // one destination (or part) per wave for the whole run
    uint32_t alone = 0;               // heaviest other destinations dealt to a workgroup of their own
    // collective; the pre/post bitmaps and chunk groups are copied into
    // `pin_in` (pinned host memory: pre, then post, then the group ids)
    uint32_t C = 0, G = 0;
    uint64_t m = 0;
    bool multi_group = false;
    char *pin_in = nullptr;
    size_t pin_in_cap = 0;
    std::vector<uint64_t> gmask;
    int op = 0;
    std::vector<uint32_t> T, slot_time;
    uint32_t tmin = 0;
    // switch model (Sec. 4.7)
    std::vector<uint32_t> sw_buf;  // per switch: buffer capacity, 0 = unlimited
    std::vector<uint8_t> sw_uni;   // per switch: 1 = no multicast
    bool sw_model = false;         // some switch has a limit or no multicast
    bool sw_built = false;         // tables below match the topology, model and chunk count
    bool sw_active = false;        // the switch-model matching kernel runs
    std::vector<uint32_t> swt;     // switch-model tables, uploaded as one region
    std::vector<uint32_t> sw_links;  // links of each switch group
    uint64_t swo[21] = {};         // offsets of the tables inside swt (order of SwTab)
    bool sw_gate = false;          // only the no-multicast rule may bind: the plain kernel runs when it cannot
    uint32_t sw_nuni = 0;          // unicast switches with out-links
    bool ran_sw = false;           // the last synthesis ran the switch-group kernel
    uint32_t sw_groups = 0, sw_pool = 0, sw_nbt = 0;
    int sw_grid = 0;
    // plan (made once per collective and switch model, before any workspace)
    bool planned = false;
    uint64_t plan_gen = 0;         // changes with every plan (static scratch ownership)
    // pinned host image of the small per-topology arrays the kernels read
    // (link and slot tables, destination deal, group masks, switch tables),
    // built by the plan; IMG_PARTS pieces at img_off[k], img_len[k] bytes
    char *pin_img = nullptr;
    size_t pin_img_cap = 0;
    size_t img_off[16] = {}, img_len[16] = {};
    uint64_t serial = 0;           // unique per context
    uint64_t static_call = 0;      // the static-scratch call whose result this context holds
    // workspace
    char *ws = nullptr;
    bool ws_static = false;        // the workspace is the library's static scratch
    size_t ws_bytes = 0;
    uint64_t max_sends = 0;
    hipStream_t stream = nullptr;
    Layout ly{};
    Sizes sz{};
    int grid = 0, wpb = 0;  // matching kernel: workgroups, waves per workgroup

    bool mirror = false;    // matching kernel keeps each destination's needs row in LDS
    // stage timing; ev[1] also marks that the setup's counts have reached `pin`
    // (events and the pinned block are made by pccl_create, so that a
    // synthesize call allocates nothing)
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    float stage_ms[3] = {0.f, 0.f, 0.f};
    // pinned host copies of the control block: [0] after the setup, [1] at the end
    Control *pin = nullptr;
    ~pccl_ctx()
    {
        (void)hipSetDevice(device);
        for (hipEvent_t e : ev)
            if (e) (void)hipEventDestroy(e);
        if (pin) (void)hipHostFree(pin);
        if (pin_in) (void)hipHostFree(pin_in);
        if (pin_img) (void)hipHostFree(pin_img);
    }
    // results
    std::unordered_map<uint64_t, uint64_t> receipt;  // (chunk << 32 | device) -> (link << 32 | t_start), copy schedule
    bool have_receipts = false;
    uint64_t n_sends = 0, n_copy = 0;
    uint32_t coll_time = 0;
    Control ctl_host{};
};

namespace {

pccl_status fail(pccl_ctx *c, pccl_status st, const char *fmt, ...) __attribute__((format(printf, 3, 4)));
pccl_status fail(pccl_ctx *c, pccl_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    return st;
}

pccl_status hip_fail(pccl_ctx *c, hipError_t e, const char *what)
{
    return fail(c, PCCL_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_OR_FAIL(ctx, expr)                                   \
    do {                                                         \
        hipError_t e_ = (expr);                                  \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr); \
    } while (0)

uint64_t words(uint64_t bits) { return (bits + 63) / 64; }

// Workspace carving: every array 256-byte aligned, in a fixed order.
struct Carver {
    char *base;
    size_t off = 0;
    template <class X>
    X *take(uint64_t count)
    {
        off = (off + 255) & ~size_t(255);
        X *p = base ? reinterpret_cast<X *>(base + off) : nullptr;
        off += sizeof(X) * (count ? count : 1);
        return p;
    }
};

void carve(pccl_ctx *c, char *base, uint64_t max_sends, Layout &ly, Sizes &sz, size_t &total)
{
    sz.N = c->N;
    sz.S = c->S;
    sz.D = c->D;
    sz.L = c->L;
    sz.C = c->C;
    sz.G = c->G;
    sz.W = words(c->C);
    sz.Wp = std::max<uint64_t>(ROW_ALIGN_WORDS, (sz.W + ROW_ALIGN_WORDS - 1) / ROW_ALIGN_WORDS * ROW_ALIGN_WORDS);
    sz.WN = words(c->N);
    sz.max_sends = max_sends;
    sz.tmin = c->tmin;
    sz.resident = c->resident ? 1u : 0u;
    sz.sw_gate = c->sw_active && c->sw_gate ? 1u : 0u;
    sz.sw_nbt = c->sw_active ? c->sw_nbt : 0u;
    const uint64_t hb = (uint64_t)sz.D * sz.Wp * sizeof(uint64_t);
    sz.hbytes = hb < (1ull << 31) ? (uint32_t)hb : 0u;
    const uint64_t nsort = std::max<uint64_t>(c->C, max_sends);
    sz.max_tiles = (uint32_t)((nsort + SORT_TILE - 1) / SORT_TILE);
    if (sz.max_tiles == 0) sz.max_tiles = 1;
    const uint64_t L = c->L, D = c->D, N = c->N, C = c->C;
    Carver cv{base};
    ly.ctl = cv.take<Control>(1);
    ly.lsrc = cv.take<uint32_t>(L);
    ly.ldst = cv.take<uint32_t>(L);
    ly.ltime = cv.take<uint32_t>(L);
    ly.lrev = cv.take<uint32_t>(L);
    ly.in_off = cv.take<uint32_t>(D + 1);
    ly.slot_link = cv.take<uint32_t>(L);
    ly.slot_src = cv.take<uint32_t>(L);
    ly.slot_time = cv.take<uint32_t>(L);
    ly.slot_cum = cv.take<uint32_t>(L);
    ly.dest_pairs = cv.take<uint32_t>(D);
    ly.group_masks = cv.take<uint64_t>((uint64_t)c->G * sz.WN);
    ly.pre = cv.take<uint64_t>(N * sz.W);
    ly.post = cv.take<uint64_t>(N * sz.W);
    ly.chunk_group = c->multi_group ? cv.take<uint16_t>(C) : nullptr;
    ly.chunk_src = cv.take<uint32_t>(C);
    ly.holder_cnt = cv.take<uint32_t>(C);
    ly.chunk_dist = cv.take<uint64_t>(C);
    ly.rank = cv.take<uint32_t>(C);
    ly.order = cv.take<uint32_t>(C);
    ly.src_index = cv.take<uint32_t>(N);
    ly.src_list = cv.take<uint32_t>(N);
    ly.sp_dist = cv.take<uint64_t>(N * D);
    ly.sp_parent = cv.take<uint32_t>(N * D);
    ly.skey[0] = cv.take<uint64_t>(nsort);
    ly.skey[1] = cv.take<uint64_t>(nsort);
    ly.sval[0] = cv.take<uint32_t>(nsort);
    ly.sval[1] = cv.take<uint32_t>(nsort);
    ly.hist = cv.take<uint32_t>(256ull * hist_stride(sz.max_tiles));
    ly.holds = cv.take<uint64_t>(D * sz.Wp);
    ly.needs = cv.take<uint64_t>(D * sz.Wp);
    ly.busy = cv.take<uint32_t>(L);
    ly.infl = cv.take<uint32_t>(L);
    ly.cur = cv.take<uint32_t>(L);
    ly.lflags = cv.take<uint32_t>(L);
    ly.lcnt = cv.take<uint32_t>(L);
    ly.snap = cv.take<uint64_t>(3 * L);
    ly.dest_log = cv.take<unsigned long long>(D);
    ly.xslot = cv.take<uint64_t>(2ull * MAX_MATCH_GRID * XSLOT_WORDS);
    ly.wave_dest = cv.take<uint32_t>(D + (uint64_t)MATCH_WAVES * MAX_MATCH_GRID);
    ly.wave_part = cv.take<uint32_t>(D + (uint64_t)MATCH_WAVES * MAX_MATCH_GRID);
    ly.out = cv.take<pccl_send>((c->op == PCCL_OP_ALLREDUCE ? 2 : 1) * max_sends);
    ly.sw = SwTab{};
    if (c->sw_active) {
        uint32_t *t = cv.take<uint32_t>(c->swt.size());
        const uint32_t **p[21] = {&ly.sw.grp,    &ly.sw.blk,     &ly.sw.blk_list, &ly.sw.lk_slot, &ly.sw.lk_dl,
                                  &ly.sw.lk_srcj, &ly.sw.lk_uni,  &ly.sw.lk_dbuf,  &ly.sw.lk_sbuf, &ly.sw.d_off,
                                  &ly.sw.s_poff, &ly.sw.p_slot,  &ly.sw.u_off,    &ly.sw.u_list,  &ly.sw.b_cap,
                                  &ly.sw.b_poff, &ly.sw.b_ooff,  &ly.sw.b_out,    &ly.sw.uc_off,  &ly.sw.uc_dst,
                                  &ly.sw.b_abs};
        for (int i = 0; i < 21; i++) *p[i] = t ? t + c->swo[i] : nullptr;
        ly.sw.pool_c = cv.take<uint32_t>(c->sw_pool);
        ly.sw.pool_n = cv.take<uint32_t>(c->sw_pool);
        ly.sw.occ = cv.take<uint32_t>(c->sw_nbt);
        ly.sw.acnt = cv.take<uint32_t>((uint64_t)c->sw_nbt * std::max<uint64_t>(C, 1));
    }
    total = (cv.off + 255) & ~size_t(255);
}

// Switch groups (Sec. 4.7 switch model): the out-neighbours of a unicast
// switch, and a limited switch with its out-neighbours, must share one
// workgroup, since their links clash on the same copy or the same buffer.
// Union-find closes those sets; each group lists its destinations' in-links
// (destination-major), the distinct sources of those links with the source's
// own in-links (where arrivals come from), its unicast switches with their
// out-links, and its limited switches with their buffer places and
// out-neighbours.  Capacities at or above the chunk count never bind and
// count as unlimited.
pccl_status build_switch_tables(pccl_ctx *c)
{
    c->sw_built = true;
    c->sw_active = false;
    c->sw_gate = false;
    c->sw_nuni = 0;
    c->swt.clear();
    c->sw_links.clear();
    if (!c->sw_model) return PCCL_OK;
    const uint32_t N = c->N, S = c->S, D = c->D, L = c->L;
    std::vector<uint32_t> cap(S);
    std::vector<uint8_t> uni(S);
    bool any = false;
    for (uint32_t i = 0; i < S; i++) {
        cap[i] = (c->sw_buf[i] && c->sw_buf[i] < c->C) ? c->sw_buf[i] : 0u;
        uni[i] = c->sw_uni[i] ? 1 : 0;
        any = any || cap[i] || uni[i];
    }
    if (!any) return PCCL_OK;
    std::vector<uint32_t> out_off(D + 1, 0), out_l(L), slot_of(L);
    for (uint32_t l = 0; l < L; l++) out_off[c->src[l] + 1]++;
    for (uint32_t v = 0; v < D; v++) out_off[v + 1] += out_off[v];
    {
        std::vector<uint32_t> fill(out_off.begin(), out_off.end() - 1);
        for (uint32_t l = 0; l < L; l++) out_l[fill[c->src[l]]++] = l;
    }
    for (uint32_t sl = 0; sl < L; sl++) slot_of[c->slot_link[sl]] = sl;
    std::vector<uint32_t> par(D);
    std::iota(par.begin(), par.end(), 0u);
    auto find = [&](uint32_t v) {
        while (par[v] != v) v = par[v] = par[par[v]];
        return v;
    };
    auto unite = [&](uint32_t a, uint32_t b) {
        a = find(a);
        b = find(b);
        if (a != b) par[std::max(a, b)] = std::min(a, b);
    };
    for (uint32_t i = 0; i < S; i++) {
        const uint32_t v = N + i;
        for (uint32_t k = out_off[v]; k < out_off[v + 1]; k++) {
            if (uni[i]) unite(c->dst[out_l[out_off[v]]], c->dst[out_l[k]]);
            if (cap[i]) unite(v, c->dst[out_l[k]]);
        }
    }
    std::vector<uint32_t> gid_of_root(D, NONE32);
    std::vector<std::vector<uint32_t>> members, limited;
    for (uint32_t v = 0; v < D; v++) {
        if (c->in_off[v + 1] == c->in_off[v]) continue;
        const uint32_t r = find(v);
        if (gid_of_root[r] == NONE32) {
            gid_of_root[r] = (uint32_t)members.size();
            members.emplace_back();
        }
        members[gid_of_root[r]].push_back(v);
    }
    limited.resize(members.size());
    for (uint32_t i = 0; i < S; i++)
        if (cap[i] && gid_of_root[find(N + i)] != NONE32) limited[gid_of_root[find(N + i)]].push_back(N + i);
    const uint32_t G = (uint32_t)members.size();
    std::vector<uint32_t> grp(16ull * G), lk_slot, lk_dl, lk_srcj, lk_uni, lk_dbuf, lk_sbuf, d_off, s_poff, p_slot,
        u_off, u_list, b_cap, b_poff, b_ooff, b_out, b_abs;
    std::vector<uint32_t> loc(L, NONE32), sidx(D, NONE32), bidx(D, NONE32), uidx(D, NONE32);
    uint32_t pool = 0;
    for (uint32_t g = 0; g < G; g++) {
        const auto &mem = members[g];
        const uint32_t lbase = (uint32_t)lk_slot.size(), dbase = (uint32_t)d_off.size();
        const uint32_t sbase = (uint32_t)s_poff.size(), pbase = (uint32_t)p_slot.size();
        const uint32_t ubase = (uint32_t)u_off.size(), ulbase = (uint32_t)u_list.size();
        const uint32_t bbase = (uint32_t)b_cap.size(), bobase = (uint32_t)b_out.size();
        uint32_t nl = 0;
        for (uint32_t dl = 0; dl < mem.size(); dl++) {
            d_off.push_back(nl);
            for (uint32_t sl = c->in_off[mem[dl]]; sl < c->in_off[mem[dl] + 1]; sl++) {
                loc[sl] = nl++;
                lk_slot.push_back(sl);
                lk_dl.push_back(dl);
            }
        }
        d_off.push_back(nl);
        std::vector<uint32_t> srcs;
        for (uint32_t i = 0; i < nl; i++) {
            const uint32_t sv = c->slot_src[lk_slot[lbase + i]];
            if (sidx[sv] == NONE32) {
                sidx[sv] = (uint32_t)srcs.size();
                srcs.push_back(sv);
            }
            lk_srcj.push_back(sidx[sv]);
        }
        uint32_t np = 0;
        for (uint32_t sv : srcs) {
            s_poff.push_back(np);
            for (uint32_t sl = c->in_off[sv]; sl < c->in_off[sv + 1]; sl++, np++) p_slot.push_back(sl);
        }
        s_poff.push_back(np);
        uint32_t nu = 0, nul = 0;
        for (uint32_t sv : srcs) {
            if (sv < N || !uni[sv - N]) continue;
            uidx[sv] = nu++;
            u_off.push_back(nul);
            for (uint32_t k = out_off[sv]; k < out_off[sv + 1]; k++, nul++) {
                const uint32_t li = loc[slot_of[out_l[k]]];
                if (li == NONE32) return fail(c, PCCL_EINTERNAL, "unicast switch %u: out-link outside its group", sv);
                u_list.push_back(li);
            }
        }
        u_off.push_back(nul);
        uint32_t nb = 0, pl = 0, no = 0;
        for (uint32_t w : limited[g]) {
            bidx[w] = nb++;
            b_cap.push_back(cap[w - N]);
            b_poff.push_back(pl);
            b_ooff.push_back(no);
            b_abs.push_back(bobase + no);
            b_abs.push_back(out_off[w + 1] - out_off[w]);
            pl += cap[w - N];
            for (uint32_t k = out_off[w]; k < out_off[w + 1]; k++, no++) {
                // the out-neighbour (an in-link from w makes it a group
                // destination) and its destination index in the group
                const uint32_t li = loc[slot_of[out_l[k]]];
                if (li == NONE32) return fail(c, PCCL_EINTERNAL, "limited switch %u: out-link outside its group", w);
                b_out.push_back(c->dst[out_l[k]] | (lk_dl[lbase + li] << 16));
            }
        }
        b_cap.push_back(0);
        b_abs.push_back(0);
        b_abs.push_back(0);
        b_poff.push_back(pl);
        b_ooff.push_back(no);
        for (uint32_t i = 0; i < nl; i++) {
            const uint32_t sl = lk_slot[lbase + i], sv = c->slot_src[sl], dv = c->dst[c->slot_link[sl]];
            lk_uni.push_back(uidx[sv]);
            lk_dbuf.push_back(bidx[dv]);
            lk_sbuf.push_back(bidx[sv]);
        }
        const uint32_t nd = (uint32_t)mem.size();
        for (uint32_t i = 0; i < nl; i++) loc[lk_slot[lbase + i]] = NONE32;
        for (uint32_t sv : srcs) {
            sidx[sv] = NONE32;
            uidx[sv] = NONE32;
        }
        for (uint32_t w : limited[g]) bidx[w] = NONE32;
        if (nl > SW_MAX_LINKS || nd > SW_MAX_LINKS)
            return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u has %u in-links (limit %u)", mem[0], nl,
                        SW_MAX_LINKS);
        if (srcs.size() > SW_MAX_SRC)
            return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u has %zu sources (limit %u)", mem[0],
                        srcs.size(), SW_MAX_SRC);
        if (np > SW_MAX_PAIRS)
            return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u: its sources have %u in-links (limit %u)",
                        mem[0], np, SW_MAX_PAIRS);
        for (uint32_t sv : srcs)
            if (c->in_off[sv + 1] - c->in_off[sv] > SW_MAX_SRC_IN)
                return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u: source %u has %u in-links (limit %u)",
                            mem[0], sv, c->in_off[sv + 1] - c->in_off[sv], SW_MAX_SRC_IN);
        if (nu > SW_MAX_SW || nb > SW_MAX_SW)
            return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u has %u unicast and %u limited switches "
                        "(limit %u each)", mem[0], nu, nb, SW_MAX_SW);
        if (pl > SW_MAX_POOL)
            return fail(c, PCCL_EUNSUPPORTED, "switch group of device %u has %u buffer places (limit %u)", mem[0], pl,
                        SW_MAX_POOL);
        const uint32_t h[16] = {nl, lbase, nd, dbase, (uint32_t)srcs.size(), sbase, np, pbase,
                                nu, ubase, ulbase, nb, bbase, bobase, pool, pl};
        std::copy(h, h + 16, grp.begin() + 16ull * g);
        pool += pl;
        c->sw_links.push_back(nl);
    }
    // the matcher indexes its snapshot entries by group link position (each
    // link is an in-link of exactly one group's destination): a pair names
    // the position of its in-link
    {
        std::vector<uint32_t> gpos(L, NONE32);
        for (uint32_t x = 0; x < (uint32_t)lk_slot.size(); x++) gpos[lk_slot[x]] = x;
        for (uint32_t &v : p_slot) {
            if (gpos[v] == NONE32) return fail(c, PCCL_EINTERNAL, "arrival pair on slot %u outside every group", v);
            v = gpos[v];
        }
    }
    // with no binding buffer limit only the no-multicast rule can change the
    // schedule, and only if two out-neighbours of one unicast switch need the
    // same chunk: the device checks that after the setup (the needs rows
    // include the relay marks) and runs the plain kernel when they never do
    std::vector<uint32_t> uc_off, uc_dst;
    bool any_cap = false;
    for (uint32_t i = 0; i < S; i++) any_cap = any_cap || cap[i];
    for (uint32_t i = 0; i < S; i++) {
        const uint32_t v = N + i;
        if (!uni[i] || out_off[v + 1] - out_off[v] < 2) continue;
        uc_off.push_back((uint32_t)uc_dst.size());
        for (uint32_t k = out_off[v]; k < out_off[v + 1]; k++) uc_dst.push_back(c->dst[out_l[k]]);
    }
    c->sw_nuni = (uint32_t)uc_off.size();
    uc_off.push_back((uint32_t)uc_dst.size());
    c->sw_gate = !any_cap;
    std::vector<const std::vector<uint32_t> *> parts = {&grp,    nullptr, nullptr, &lk_slot, &lk_dl,  &lk_srcj,
                                                        &lk_uni, &lk_dbuf, &lk_sbuf, &d_off,  &s_poff, &p_slot,
                                                        &u_off,  &u_list,  &b_cap,   &b_poff, &b_ooff, &b_out,
                                                        &uc_off, &uc_dst,  &b_abs};
    uint64_t off = 0;
    for (int i = 0; i < 21; i++) {
        c->swo[i] = off;
        off += i == 1 ? MAX_MATCH_GRID + 1ull : i == 2 ? (uint64_t)G : parts[i]->size();
        off = (off + 63) & ~63ull;
    }
    c->swt.assign(off, 0u);
    for (int i = 0; i < 21; i++)
        if (parts[i]) std::copy(parts[i]->begin(), parts[i]->end(), c->swt.begin() + c->swo[i]);
    c->sw_groups = G;
    c->sw_pool = pool;
    c->sw_nbt = (uint32_t)b_cap.size();
    c->sw_active = true;
    return PCCL_OK;
}

// Switch groups to workgroups: heaviest first, dealt round-robin.
pccl_status deal_switch_groups(pccl_ctx *c)
{
    const uint32_t G = c->sw_groups, nb = (uint32_t)c->sw_grid;
    std::vector<uint32_t> byweight(G);
    std::iota(byweight.begin(), byweight.end(), 0u);
    std::stable_sort(byweight.begin(), byweight.end(),
                     [&](uint32_t a, uint32_t b) { return c->sw_links[a] > c->sw_links[b]; });
    uint32_t *blk = c->swt.data() + c->swo[1], *list = c->swt.data() + c->swo[2];
    uint32_t k = 0;
    for (uint32_t b = 0; b < nb; b++) {
        blk[b] = k;
        uint64_t links = 0;
        for (uint32_t i = b; i < G; i += nb) {
            list[k++] = byweight[i];
            links += c->sw_links[byweight[i]];
        }
        if (links >= (1u << 19))
            return fail(c, PCCL_EUNSUPPORTED, "switch-model workgroup %u would own %llu links", b,
                        (unsigned long long)links);
    }
    blk[nb] = k;
    return PCCL_OK;
}

// Destinations of the matching kernel's waves.  Split destinations first,
// each taking a whole workgroup (wave p is part p; parts past the last are
// empty and only take part in the part barriers).  The others heaviest first
// (most arrival pairs, then most in-links), dealt across the remaining
// workgroups before filling any workgroup's second wave, so that heavy
// destinations do not share a compute unit and its memory pipeline.  Pass r
// of wave w handles entry r * nwaves + w.
void deal_destinations(pccl_ctx *c)
{
    const uint32_t D = c->D, nb = (uint32_t)c->grid, wpb = (uint32_t)c->wpb, nw = nb * wpb;
    std::vector<uint8_t> is_split(D, 0);
    for (uint32_t d : c->split) is_split[d] = 1;
    std::vector<uint32_t> byweight;
    byweight.reserve(D);
    for (uint32_t v = 0; v < D; v++)
        if (!is_split[v]) byweight.push_back(v);
    std::stable_sort(byweight.begin(), byweight.end(), [&](uint32_t a, uint32_t b) {
        if (c->dest_pairs[a] != c->dest_pairs[b]) return c->dest_pairs[a] > c->dest_pairs[b];
        return c->in_off[a + 1] - c->in_off[a] > c->in_off[b + 1] - c->in_off[b];
    });
    // the `alone` heaviest unsplit destinations take wave 0 of the next
    // workgroups (one pass, by construction of the grid)
    const uint32_t hs = (uint32_t)c->split.size(), ha = c->alone, h = hs + ha;
    const uint32_t nb2 = nb - h, rest = (uint32_t)byweight.size() - ha;
    const uint32_t n2 = nb2 * wpb;
    const uint32_t passes = n2 ? std::max(1u, (rest + n2 - 1) / n2) : 1u;
    c->wave_dest.assign((size_t)passes * nw, NONE32);
    c->wave_part.assign((size_t)passes * nw, 0u);
    for (uint32_t i = 0; i < hs; i++) {
        const uint32_t d = c->split[i];
        const std::vector<uint32_t> &cut = c->split_cuts[i];  // cut[p] = first in-link of part p; cut.back() = in-degree
        const uint32_t parts = (uint32_t)cut.size() - 1;
        for (uint32_t p = 0; p < wpb; p++) {
            const uint32_t first = p < parts ? cut[p] : cut.back(), cnt = p < parts ? cut[p + 1] - cut[p] : 0u;
            c->wave_dest[(size_t)i * wpb + p] = d;
            c->wave_part[(size_t)i * wpb + p] = (wpb << 24) | (p << 16) | (first << 8) | cnt;
        }
    }
    for (uint32_t i = 0; i < ha; i++) c->wave_dest[(size_t)(hs + i) * wpb] = byweight[i];
    for (uint32_t q = 0; q < rest; q++) {
        const uint32_t r = q / n2, j = q % n2, w = (h + j % nb2) * wpb + j / nb2;
        c->wave_dest[(size_t)r * nw + w] = byweight[ha + q];
    }
}

uint64_t safe_max_sends(const pccl_ctx *c)
{
    return (uint64_t)c->C * (c->D > 0 ? c->D - 1 : 0);
}

const char *einval_detail(uint32_t code)
{
    switch (code) {
    case 1: return "a bit is set beyond the last chunk";
    case 2: return "a pre/postcondition bit sits on an NPU outside the chunk's process group";
    case 3: return "chunk group id out of range";
    case 4: return "chunk has more than one precondition holder";
    case 5: return "chunk is needed by a postcondition but held by no NPU";
    default: return "invalid collective";
    }
}

uint64_t row_words(uint32_t C)
{
    const uint64_t W = words(C);
    return std::max<uint64_t>(ROW_ALIGN_WORDS, (W + ROW_ALIGN_WORDS - 1) / ROW_ALIGN_WORDS * ROW_ALIGN_WORDS);
}

// Pinned host memory of at least `bytes` in *buf (grown, never shrunk).
pccl_status ensure_pinned(pccl_ctx *c, char **buf, size_t *cap, size_t bytes)
{
    if (*cap >= bytes && *buf) return PCCL_OK;
    if (*buf) {
        (void)hipHostFree(*buf);
        *buf = nullptr;
        *cap = 0;
    }
    const size_t n = std::max<size_t>(bytes, 256);
    HIP_OR_FAIL(c, hipHostMalloc((void **)buf, n, hipHostMallocDefault));
    *cap = n;
    return PCCL_OK;
}

constexpr int IMG_PARTS = 14;

// Parts of destination d for a split over the waves of a workgroup:
// consecutive in-links, at most `target` links and MAX_PAIRS arrival pairs
// per part (MAX_IN_LINKS links at most).  Returns the first in-link of each
// part followed by the in-degree.
std::vector<uint32_t> cut_parts(const pccl_ctx *c, uint32_t d, uint32_t target)
{
    std::vector<uint32_t> cut = {0};
    const uint32_t b = c->in_off[d], n = c->in_off[d + 1] - b;
    target = std::min<uint32_t>(std::max<uint32_t>(target, 1), MAX_IN_LINKS);
    uint32_t links = 0, pairs = 0;
    for (uint32_t i = 0; i < n; i++) {
        const uint32_t s = c->slot_src[b + i], p = c->in_off[s + 1] - c->in_off[s];
        if (links == target || pairs + p > MAX_PAIRS) {
            cut.push_back(i);
            links = pairs = 0;
        }
        links++;
        pairs += p;
    }
    cut.push_back(n);
    return cut;
}

// Everything that depends on the topology, the collective and the switch
// model but not on the workspace: the switch tables, the matching kernel's
// launch shape (waves per workgroup, needs rows in LDS, grid), the deal of
// destinations to waves and the pinned image of the small arrays the kernels
// read.  Made when the collective or the switch model is set, so that binding
// a workspace only carves it and a synthesize call allocates nothing.
pccl_status plan(pccl_ctx *c)
{
    c->planned = false;
    c->have_ws = c->uploaded = c->have_result = false;
    pccl_status st = build_switch_tables(c);
    if (st != PCCL_OK) return st;
    HIP_OR_FAIL(c, hipSetDevice(c->device));
    const uint64_t Wp = row_words(c->C);
    const uint64_t hb = (uint64_t)c->D * Wp * sizeof(uint64_t);
    const bool desc_ok = hb < (1ull << 31);  // the LDS-row kernel reads holds through one buffer descriptor
    // destinations one wave cannot take (more than MAX_IN_LINKS in-links or
    // MAX_PAIRS arrival pairs) are split over the waves of one workgroup
    std::vector<uint32_t> must;
    uint32_t need_w = 1;
    for (uint32_t d = 0; d < c->D; d++) {
        const uint32_t parts = (uint32_t)cut_parts(c, d, MAX_IN_LINKS).size() - 1;
        if (parts > 1) {
            must.push_back(d);
            need_w = std::max(need_w, parts);
        }
    }
    if (need_w > MATCH_WAVES)
        return fail(c, PCCL_EUNSUPPORTED, "a device needs %u waves for its in-links and arrival pairs (limit %u)", need_w,
                    MATCH_WAVES);
    // heavy destinations (at least four times the mean arrival pairs) get a
    // workgroup, so a compute unit, of their own when the grid has room for
    // it: their wave then has the unit's memory pipeline and LDS to itself
    uint32_t n_heavy = 0;
    {
        uint64_t tot = 0;
        for (uint32_t v = 0; v < c->D; v++) tot += c->dest_pairs[v];
        std::vector<uint8_t> is_must(c->D, 0);
        for (uint32_t d : must) is_must[d] = 1;
        for (uint32_t v = 0; v < c->D; v++)
            if (!is_must[v] && c->dest_pairs[v] > 0 && (uint64_t)c->dest_pairs[v] * c->D >= 4 * tot) n_heavy++;
    }
    const uint32_t D1 = std::max<uint32_t>(c->D, 1);
    // the grid for w waves per workgroup with at most gmax workgroups:
    // split destinations take a workgroup each, heavy ones too if it fits,
    // the others a wave each
    auto shape = [&](uint32_t w, int gmax, int &grid, bool &resident, uint32_t &alone) {
        const uint64_t ns = must.size();
        alone = 0;
        const uint64_t g0 = ns + ((uint64_t)c->D - ns + w - 1) / w;
        if (g0 > (uint64_t)gmax) {
            if (ns) return false;
            grid = std::min<int>(gmax, (int)((D1 + w - 1) / w));
            resident = (uint64_t)grid * w >= c->D;
            return grid > 0;
        }
        grid = (int)std::max<uint64_t>(g0, 1);
        resident = true;
        if (w > 1 && n_heavy) {
            const uint64_t g1 = ns + n_heavy + ((uint64_t)c->D - ns - n_heavy + w - 1) / w;
            if (g1 <= (uint64_t)gmax) {
                alone = n_heavy;
                grid = (int)g1;
            }
        }
        return true;
    };
    // waves per workgroup: as few as keep the grid near MATCH_TARGET_GRID
    // workgroups, so that few destinations still spread over many compute
    // units while many destinations do not make the window exchange poll
    // too many slots; at least as many as the largest split destination has
    // parts
    int wpb = (int)std::min<uint32_t>(MATCH_WAVES, std::max<uint32_t>(1, (D1 + MATCH_TARGET_GRID - 1) / MATCH_TARGET_GRID));
    wpb = std::max<int>(wpb, (int)need_w);
    // needs rows in LDS: with as many of those waves as leave room for one
    // row per wave, when every wave then owns one destination (or part)
    c->mirror = false;
    int lds_cu = 0;
    HIP_OR_FAIL(c, hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, c->device));
    const size_t lds_static = match_static_lds(), row_bytes = (size_t)Wp * sizeof(uint64_t);
    const bool spl = !must.empty();
    int grid = 0;
    bool resident = false;
    uint32_t alone = 0;
    for (int w = wpb; w >= (int)need_w && lds_static > 0 && desc_ok; w--) {
        const size_t dyn = (size_t)w * row_bytes;
        if (lds_static + dyn > (size_t)lds_cu) continue;
        const int gmax = std::min<int>(match_max_grid(c->device, w, true, dyn, spl), (int)MAX_MATCH_GRID);
        if (gmax > 0 && shape((uint32_t)w, gmax, grid, resident, alone) && resident) {
            wpb = w;
            c->mirror = true;
            break;
        }
    }
    if (!c->mirror) {
        const int gmax = std::min<int>(match_max_grid(c->device, wpb, false, 0, spl), (int)MAX_MATCH_GRID);
        if (gmax <= 0) return fail(c, PCCL_EDEVICE, "matching kernel cannot be resident");
        if (!shape((uint32_t)wpb, gmax, grid, resident, alone))
            return fail(c, PCCL_EUNSUPPORTED, "device %u needs %u waves for its in-links and arrival pairs; the "
                        "matching kernel cannot keep a workgroup per such device and a wave per other device "
                        "resident (%d workgroups of %d waves at most)", must[0], need_w, gmax, wpb);
    }
    c->wpb = wpb;
    c->grid = grid;
    c->resident = resident;
    c->alone = alone;
    c->split = must;
    c->split_cuts.clear();
    for (uint32_t d : c->split) {
        // the in-links spread evenly over the workgroup's waves (as few
        // parts as fit when the pairs do not allow that)
        const uint32_t n = c->in_off[d + 1] - c->in_off[d];
        std::vector<uint32_t> cut = cut_parts(c, d, (n + wpb - 1) / wpb);
        if (cut.size() - 1 > (size_t)wpb) cut = cut_parts(c, d, MAX_IN_LINKS);
        c->split_cuts.push_back(cut);
    }
    deal_destinations(c);
    if (c->sw_active) {
        c->sw_grid = std::min<int>(std::min<int>(match_sw_max_grid(c->device), (int)MAX_MATCH_GRID),
                                   (int)c->sw_groups);
        if (c->sw_grid <= 0) return fail(c, PCCL_EDEVICE, "switch-model matching kernel cannot be resident");
        st = deal_switch_groups(c);
        if (st != PCCL_OK) return st;
    }
    // the pinned image, in the order upload() copies it
    const std::pair<const void *, size_t> parts[IMG_PARTS] = {
        {c->src.data(), 4ull * c->L},         {c->dst.data(), 4ull * c->L},
        {c->T.data(), 4ull * c->L},           {c->rev.data(), 4ull * c->L},
        {c->in_off.data(), 4ull * (c->D + 1)}, {c->slot_link.data(), 4ull * c->L},
        {c->slot_src.data(), 4ull * c->L},    {c->slot_time.data(), 4ull * c->L},
        {c->slot_cum.data(), 4ull * c->L},    {c->dest_pairs.data(), 4ull * c->D},
        {c->wave_dest.data(), 4ull * c->wave_dest.size()},
        {c->wave_part.data(), 4ull * c->wave_part.size()},
        {c->gmask.data(), 8ull * c->gmask.size()},
        {c->swt.data(), c->sw_active ? 4ull * c->swt.size() : 0ull}};
    size_t total = 0;
    for (int k = 0; k < IMG_PARTS; k++) {
        c->img_off[k] = total;
        c->img_len[k] = parts[k].second;
        total += (parts[k].second + 255) & ~size_t(255);
    }
    st = ensure_pinned(c, &c->pin_img, &c->pin_img_cap, total);
    if (st != PCCL_OK) return st;
    for (int k = 0; k < IMG_PARTS; k++)
        if (c->img_len[k]) std::memcpy(c->pin_img + c->img_off[k], parts[k].first, c->img_len[k]);
    c->planned = true;
    c->plan_gen++;
    return PCCL_OK;
}

// Points the context at a workspace: carves the layout for `max_sends`
// transfers.  The inputs are copied in by the next synthesize call.
pccl_status bind_workspace(pccl_ctx *c, char *ptr, size_t bytes, uint64_t ms, hipStream_t st, bool is_static)
{
    Layout ly{};
    Sizes sz{};
    size_t need = 0;
    carve(c, nullptr, ms, ly, sz, need);
    if (bytes < need) {
        if (is_static)
            return fail(c, PCCL_ENOMEM, "the library's static scratch holds %zu bytes, this collective needs %zu "
                        "(pass a tighter max_sends, or bring a workspace with pccl_set_workspace)", bytes, need);
        return fail(c, PCCL_ENOMEM, "workspace has %zu bytes, needs %zu", bytes, need);
    }
    carve(c, ptr, ms, c->ly, c->sz, need);
    c->ws = ptr;
    c->ws_bytes = bytes;
    c->max_sends = ms;
    c->stream = st;
    c->ws_static = is_static;
    c->have_ws = true;
    c->uploaded = c->have_result = false;
    return PCCL_OK;
}

constexpr int MAX_SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[MAX_SCRATCH_DEVICES] = {};
// Whose inputs each device's scratch holds (context serial, plan generation,
// max_sends; serial 0 = nobody's), so that repeated calls of one context
// skip the copy, and the number of the last call, so that a context whose
// result a later call overwrote is told so.
struct ScratchOwner {
    uint64_t serial, plan_gen, max_sends, call;
};
ScratchOwner g_scratch_owner[MAX_SCRATCH_DEVICES] = {};
uint64_t g_next_serial = 1;

// The context's schedule is still in its workspace (a result in the static
// scratch is gone once another call used the scratch).
bool result_alive(const pccl_ctx *c)
{
    if (!c->have_result) return false;
    if (!c->ws_static) return true;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    const ScratchOwner &o = g_scratch_owner[c->device];
    return o.call == c->static_call && o.serial == c->serial;
}

}  // namespace

#define GUARD_BEGIN try {
#define GUARD_END(ctx)                                                   \
    }                                                                    \
    catch (const std::exception &ex)                                     \
    {                                                                    \
        return fail((ctx), PCCL_EINTERNAL, "exception: %s", ex.what()); \
    }                                                                    \
    catch (...)                                                          \
    {                                                                    \
        return fail((ctx), PCCL_EINTERNAL, "unknown exception");         \
    }

extern "C" {

pccl_status pccl_create(pccl_ctx **out, int hip_device, uint64_t tie_seed)
{
    if (!out) return PCCL_EINVAL;
    *out = nullptr;
    GUARD_BEGIN
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || hip_device < 0 || hip_device >= n) return PCCL_EDEVICE;
    if (hipSetDevice(hip_device) != hipSuccess) return PCCL_EDEVICE;
    if (hip_device >= MAX_SCRATCH_DEVICES) return PCCL_EDEVICE;
    {
        // this device's copy of the static scratch, looked up once
        std::lock_guard<std::mutex> g(g_scratch_mu);
        if (!g_scratch_ptr[hip_device]) {
            void *ptr = nullptr;
            if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return PCCL_EDEVICE;
            g_scratch_ptr[hip_device] = ptr;
        }
    }
    pccl_ctx *c = new pccl_ctx();
    c->device = hip_device;
    c->seed = tie_seed;
    {
        std::lock_guard<std::mutex> g(g_scratch_mu);
        c->serial = g_next_serial++;
    }
    // the stage events and the pinned control-block copies, made here so
    // that synthesize calls allocate nothing
    bool ok = hipHostMalloc((void **)&c->pin, 2 * sizeof(Control), hipHostMallocDefault) == hipSuccess;
    for (hipEvent_t &e : c->ev) ok = ok && hipEventCreate(&e) == hipSuccess;
    if (!ok) {
        delete c;
        return PCCL_EDEVICE;
    }
    *out = c;
    return PCCL_OK;
    GUARD_END(nullptr)
}

void pccl_destroy(pccl_ctx *ctx) { delete ctx; }

const char *pccl_last_error(const pccl_ctx *ctx) { return ctx ? ctx->err.c_str() : "null context"; }

pccl_status pccl_load_topology(pccl_ctx *c, uint32_t n_npus, uint32_t n_switches, uint32_t n_links,
                               const uint32_t *link_src, const uint32_t *link_dst, const uint32_t *alpha_ns,
                               const uint32_t *bw_GBps)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    if (n_npus == 0) return fail(c, PCCL_EINVAL, "no NPUs");
    if (n_links && (!link_src || !link_dst || !alpha_ns || !bw_GBps)) return fail(c, PCCL_EINVAL, "null link array");
    const uint64_t D64 = (uint64_t)n_npus + n_switches;
    if (D64 > MAX_DEVICES_SP) return fail(c, PCCL_EUNSUPPORTED, "%llu devices (limit %u)", (unsigned long long)D64, MAX_DEVICES_SP);
    const uint32_t D = (uint32_t)D64, L = n_links;
    if (L >= (1u << 24)) return fail(c, PCCL_EUNSUPPORTED, "%u links (limit 2^24 - 1)", L);
    std::unordered_map<uint64_t, uint32_t> seen;
    seen.reserve(L * 2 + 1);
    for (uint32_t l = 0; l < L; l++) {
        if (link_src[l] >= D || link_dst[l] >= D) return fail(c, PCCL_EINVAL, "link %u endpoint out of range", l);
        if (link_src[l] == link_dst[l]) return fail(c, PCCL_EINVAL, "link %u is a self loop", l);
        if (bw_GBps[l] == 0) return fail(c, PCCL_EINVAL, "link %u has zero bandwidth", l);
        const uint64_t key = ((uint64_t)link_src[l] << 32) | link_dst[l];
        auto it = seen.find(key);
        if (it != seen.end()) return fail(c, PCCL_EINVAL, "links %u and %u are duplicates", it->second, l);
        seen.emplace(key, l);
    }
    // destination-major slots
    std::vector<uint32_t> in_off(D + 1, 0), fill(D, 0), slot_link(L), slot_src(L), slot_cum(L), dest_pairs(D, 0);
    for (uint32_t l = 0; l < L; l++) in_off[link_dst[l] + 1]++;
    for (uint32_t v = 0; v < D; v++) in_off[v + 1] += in_off[v];
    for (uint32_t l = 0; l < L; l++) {
        const uint32_t d = link_dst[l], sl = in_off[d] + fill[d]++;
        slot_link[sl] = l;
        slot_src[sl] = link_src[l];
    }
    for (uint32_t d = 0; d < D; d++) {
        const uint32_t indeg = in_off[d + 1] - in_off[d];
        if (indeg > MAX_SPLIT_LINKS)
            return fail(c, PCCL_EUNSUPPORTED, "device %u has %u in-links (limit %u)", d, indeg, MAX_SPLIT_LINKS);
        uint64_t cum = 0;
        for (uint32_t sl = in_off[d]; sl < in_off[d + 1]; sl++) {
            slot_cum[sl] = (uint32_t)cum;
            const uint32_t s = slot_src[sl];
            if (in_off[s + 1] - in_off[s] > MAX_PAIRS)
                return fail(c, PCCL_EUNSUPPORTED, "device %u has %u in-links and feeds device %u (limit %u)", s,
                            in_off[s + 1] - in_off[s], d, MAX_PAIRS);
            cum += in_off[s + 1] - in_off[s];
        }
        if (cum > (uint64_t)MATCH_WAVES * MAX_PAIRS)
            return fail(c, PCCL_EUNSUPPORTED, "device %u: its in-links' sources have %llu in-links in total (limit %u)",
                        d, (unsigned long long)cum, MATCH_WAVES * MAX_PAIRS);
        dest_pairs[d] = (uint32_t)cum;
    }
    std::vector<uint32_t> rev(L, NONE32);
    for (uint32_t l = 0; l < L; l++) {
        auto it = seen.find(((uint64_t)link_dst[l] << 32) | link_src[l]);
        if (it != seen.end()) rev[l] = it->second;
    }
    c->N = n_npus;
    c->S = n_switches;
    c->D = D;
    c->L = L;
    c->src.assign(link_src, link_src + L);
    c->dst.assign(link_dst, link_dst + L);
    c->alpha.assign(alpha_ns, alpha_ns + L);
    c->bw.assign(bw_GBps, bw_GBps + L);
    c->in_off.swap(in_off);
    c->slot_link.swap(slot_link);
    c->slot_src.swap(slot_src);
    c->slot_cum.swap(slot_cum);
    c->dest_pairs.swap(dest_pairs);
    c->rev.swap(rev);
    c->sw_buf.assign(n_switches, 0u);
    c->sw_uni.assign(n_switches, 0u);
    c->sw_model = c->sw_built = c->sw_active = false;
    c->have_topo = true;
    c->have_coll = c->planned = c->have_ws = c->uploaded = c->have_result = false;
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_set_collective(pccl_ctx *c, uint32_t n_chunks, uint64_t chunk_bytes, const uint64_t *pre_bits,
                                const uint64_t *post_bits, const uint64_t *group_masks, uint32_t n_groups,
                                const uint16_t *chunk_group, pccl_op op)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    if (!c->have_topo) return fail(c, PCCL_ESTATE, "load a topology first");
    if (chunk_bytes == 0) return fail(c, PCCL_EINVAL, "chunk size 0");
    if (n_groups == 0 || !group_masks) return fail(c, PCCL_EINVAL, "no process group");
    if (n_groups > 1 && !chunk_group) return fail(c, PCCL_EINVAL, "several groups need chunk_group");
    if (n_groups > 65536) return fail(c, PCCL_EINVAL, "too many groups");
    if (n_chunks && (!pre_bits || !post_bits)) return fail(c, PCCL_EINVAL, "null pre/post bitmap");
    if (op != PCCL_OP_COPY && op != PCCL_OP_REDUCE_REVERSED && op != PCCL_OP_ALLREDUCE)
        return fail(c, PCCL_EINVAL, "unknown op %d", (int)op);
    if ((uint64_t)n_chunks + ROW_ALIGN_WORDS * 64ull >= 0xFFFFFFFFull)
        return fail(c, PCCL_EUNSUPPORTED, "too many chunks");
    const uint64_t WN = words(c->N);
    for (uint32_t g = 0; g < n_groups; g++)
        for (uint64_t v = c->N; v < WN * 64; v++)
            if ((group_masks[g * WN + v / 64] >> (v % 64)) & 1ull)
                return fail(c, PCCL_EINVAL, "group %u names a non-NPU", g);
    std::vector<uint32_t> T(c->L);
    uint32_t tmin = NONE32;
    for (uint32_t l = 0; l < c->L; l++) {
        const uint64_t beta = chunk_bytes / c->bw[l] + (chunk_bytes % c->bw[l] != 0);
        const uint64_t t = (uint64_t)c->alpha[l] + beta;
        if (beta > 0xFFFFFFFFull || t > 0xFFFFFFFFull)
            return fail(c, PCCL_ERANGE, "link %u time does not fit in 32 bits", l);
        T[l] = (uint32_t)t;
        tmin = std::min(tmin, T[l]);
    }
    if (op != PCCL_OP_COPY) {
        for (uint32_t l = 0; l < c->L; l++)
            if (c->rev[l] == NONE32 || T[c->rev[l]] != T[l])
                return fail(c, PCCL_EUNSUPPORTED, "link %u has no reverse link of equal time", l);
    }
    // the caller's arrays are copied now (host or device memory), so they may
    // be freed on return
    const bool multi = n_groups > 1;
    const size_t bm = (size_t)c->N * words(n_chunks) * sizeof(uint64_t);
    const size_t cgb = multi ? (size_t)n_chunks * sizeof(uint16_t) : 0;
    c->have_coll = c->planned = false;
    c->have_ws = c->uploaded = c->have_result = false;
    pccl_status st = ensure_pinned(c, &c->pin_in, &c->pin_in_cap, 2 * bm + cgb);
    if (st != PCCL_OK) return st;
    HIP_OR_FAIL(c, hipSetDevice(c->device));
    if (bm) {
        HIP_OR_FAIL(c, hipMemcpy(c->pin_in, pre_bits, bm, hipMemcpyDefault));
        HIP_OR_FAIL(c, hipMemcpy(c->pin_in + bm, post_bits, bm, hipMemcpyDefault));
    }
    if (cgb) HIP_OR_FAIL(c, hipMemcpy(c->pin_in + 2 * bm, chunk_group, cgb, hipMemcpyDefault));
    std::vector<uint32_t> slot_time(c->L);
    for (uint32_t sl = 0; sl < c->L; sl++) slot_time[sl] = T[c->slot_link[sl]];
    c->C = n_chunks;
    c->m = chunk_bytes;
    c->G = n_groups;
    c->multi_group = multi;
    c->gmask.assign(group_masks, group_masks + (size_t)n_groups * WN);
    c->op = op;
    c->T.swap(T);
    c->slot_time.swap(slot_time);
    c->tmin = c->L ? tmin : 1;
    c->have_coll = true;
    return plan(c);
    GUARD_END(c)
}

pccl_status pccl_set_switch_model(pccl_ctx *c, uint32_t n_switches, const uint32_t *buffer_chunks,
                                  const uint8_t *unicast)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    if (!c->have_topo) return fail(c, PCCL_ESTATE, "load a topology first");
    if (n_switches != c->S)
        return fail(c, PCCL_EINVAL, "switch model for %u switches, topology has %u", n_switches, c->S);
    bool any = false;
    for (uint32_t i = 0; i < c->S; i++) {
        c->sw_buf[i] = buffer_chunks ? buffer_chunks[i] : 0u;
        c->sw_uni[i] = unicast ? (unicast[i] != 0) : 0u;
        any = any || c->sw_buf[i] || c->sw_uni[i];
    }
    c->sw_model = any;
    c->sw_built = c->sw_active = false;
    c->have_ws = c->uploaded = c->have_result = false;
    return c->have_coll ? plan(c) : PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_workspace_bytes(pccl_ctx *c, uint64_t max_sends, size_t *out_bytes)
{
    if (!c || !out_bytes) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!c->have_coll) return fail(c, PCCL_ESTATE, "set a collective first");
    if (!c->planned) return fail(c, PCCL_ESTATE, "the last pccl_set_collective / pccl_set_switch_model failed");
    Layout ly{};
    Sizes sz{};
    size_t total = 0;
    carve(c, nullptr, max_sends ? max_sends : safe_max_sends(c), ly, sz, total);
    *out_bytes = total;
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_set_workspace(pccl_ctx *c, void *device_ptr, size_t bytes, uint64_t max_sends, void *hip_stream)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    if (!c->have_coll) return fail(c, PCCL_ESTATE, "set a collective first");
    if (!c->planned) return fail(c, PCCL_ESTATE, "the last pccl_set_collective / pccl_set_switch_model failed");
    if (!device_ptr) return fail(c, PCCL_EINVAL, "null workspace");
    if (reinterpret_cast<uintptr_t>(device_ptr) & 255u) return fail(c, PCCL_EINVAL, "workspace not 256-byte aligned");
    c->have_ws = false;
    return bind_workspace(c, static_cast<char *>(device_ptr), bytes, max_sends ? max_sends : safe_max_sends(c),
                          static_cast<hipStream_t>(hip_stream), false);
    GUARD_END(c)
}

// Copies the plan's pinned image and the collective's inputs into the
// workspace (pinned sources: plain DMA, no staging by the runtime).
static pccl_status upload(pccl_ctx *c)
{
    const Layout &ly = c->ly;
    hipStream_t st = c->stream;
    void *dst[IMG_PARTS] = {ly.lsrc,      ly.ldst,     ly.ltime,      ly.lrev,      ly.in_off,
                            ly.slot_link, ly.slot_src, ly.slot_time,  ly.slot_cum,  ly.dest_pairs,
                            ly.wave_dest, ly.wave_part, ly.group_masks, const_cast<uint32_t *>(ly.sw.grp)};
    for (int k = 0; k < IMG_PARTS; k++)
        if (c->img_len[k])
            HIP_OR_FAIL(c, hipMemcpyAsync(dst[k], c->pin_img + c->img_off[k], c->img_len[k], hipMemcpyHostToDevice, st));
    const size_t bm = (size_t)c->N * c->sz.W * sizeof(uint64_t);
    if (bm) {
        HIP_OR_FAIL(c, hipMemcpyAsync(ly.pre, c->pin_in, bm, hipMemcpyHostToDevice, st));
        HIP_OR_FAIL(c, hipMemcpyAsync(ly.post, c->pin_in + bm, bm, hipMemcpyHostToDevice, st));
    }
    if (ly.chunk_group && c->C)
        HIP_OR_FAIL(c, hipMemcpyAsync(ly.chunk_group, c->pin_in + 2 * bm, (size_t)c->C * sizeof(uint16_t),
                                      hipMemcpyHostToDevice, st));
    c->uploaded = true;
    return PCCL_OK;
}

static pccl_status device_error(pccl_ctx *c, const Control &h)
{
    switch (h.error) {
    case ST_EINVAL:
        return fail(c, PCCL_EINVAL, "%s (chunk %u, NPU %u)", einval_detail(h.error_arg[2]), h.error_arg[0],
                    h.error_arg[1]);
    case ST_EUNREACHABLE:
        return fail(c, PCCL_EUNREACHABLE, "chunk %u: NPU %u is unreachable from NPU %u", h.error_arg[0],
                    h.error_arg[1], h.error_arg[2]);
    case ST_ERANGE:
        return fail(c, PCCL_ERANGE, "chunk %u at device %u: %s does not fit in 32 bits", h.error_arg[0],
                    h.error_arg[1], h.error_arg[2] == 1 ? "distance" : "time");
    case ST_ENOMEM:
        return fail(c, PCCL_ENOMEM, "collective needs %llu transfers, workspace holds %llu",
                    (unsigned long long)h.needs_total, (unsigned long long)h.max_sends);
    case ST_EDEADLOCK:
        return fail(c, PCCL_EDEADLOCK, "%u deliveries remain but nothing is in flight", h.error_arg[0]);
    default:
        return fail(c, PCCL_EINTERNAL, "device error %u (%u %u %u)", h.error, h.error_arg[0], h.error_arg[1],
                    h.error_arg[2]);
    }
}

// The synthesis on the bound workspace.  Allocates nothing: the events and
// the pinned control-block copies come from pccl_create, the inputs from the
// pinned staging of pccl_set_collective and the plan.
static pccl_status synthesize_bound(pccl_ctx *c, uint64_t *n_sends, uint32_t *collective_time_ns)
{
    c->have_result = false;
    HIP_OR_FAIL(c, hipSetDevice(c->device));
    hipStream_t st = c->stream;
    HIP_OR_FAIL(c, hipEventRecord(c->ev[0], st));
    if (!c->uploaded) {
        pccl_status s = upload(c);
        if (s != PCCL_OK) return s;
    }
    HIP_OR_FAIL(c, launch_setup(c->ly, c->sz, c->ly.pre, c->ly.post, c->ly.chunk_group, c->seed, st));
    // the setup's delivery count sizes the output stage; the host reads it
    // while the matching kernel runs and queues the output kernels behind it
    HIP_OR_FAIL(c, hipMemcpyAsync(&c->pin[0], c->ly.ctl, sizeof(Control), hipMemcpyDeviceToHost, st));
    HIP_OR_FAIL(c, hipEventRecord(c->ev[1], st));
    const bool gate = c->sw_active && c->sw_gate;
    if (gate) {
        // both kernels are queued; the check picks the one that runs and the
        // other returns at once
        if (c->sw_nuni) HIP_OR_FAIL(c, launch_unicast_check(c->ly, c->sz, st, c->sw_nuni));
        HIP_OR_FAIL(c, launch_match_sw(c->ly, c->sz, st, c->sw_grid));
        HIP_OR_FAIL(c, launch_match(c->ly, c->sz, st, c->grid, c->wpb, c->mirror, !c->split.empty()));
    } else if (c->sw_active) {
        HIP_OR_FAIL(c, launch_match_sw(c->ly, c->sz, st, c->sw_grid));
    } else {
        HIP_OR_FAIL(c, launch_match(c->ly, c->sz, st, c->grid, c->wpb, c->mirror, !c->split.empty()));
    }
    HIP_OR_FAIL(c, hipEventRecord(c->ev[2], st));
    HIP_OR_FAIL(c, hipEventSynchronize(c->ev[1]));
    const Control s0 = c->pin[0];
    const bool out_queued = !s0.error && s0.needs_total <= c->max_sends;
    if (out_queued) HIP_OR_FAIL(c, launch_output(c->ly, c->sz, c->op, s0.needs_total, st));
    HIP_OR_FAIL(c, hipEventRecord(c->ev[3], st));
    HIP_OR_FAIL(c, hipMemcpyAsync(&c->pin[1], c->ly.ctl, sizeof(Control), hipMemcpyDeviceToHost, st));
    HIP_OR_FAIL(c, hipStreamSynchronize(st));
    c->ctl_host = c->pin[1];
    const Control &h = c->ctl_host;
    c->ran_sw = c->sw_active && (!gate || h.sw_binds);
    if (h.abort) return fail(c, PCCL_EINTERNAL, "matching kernel barrier timed out");
    if (h.error) return device_error(c, h);
    if (h.n_log != h.needs_total || !out_queued || h.needs_total != s0.needs_total)
        return fail(c, PCCL_EINTERNAL, "logged %llu transfers for %llu deliveries", (unsigned long long)h.n_log,
                    (unsigned long long)h.needs_total);
    const uint64_t n = h.n_log;
    if (c->op == PCCL_OP_ALLREDUCE && 2ull * h.cstar > 0xFFFFFFFFull)
        return fail(c, PCCL_ERANGE, "all-reduce time does not fit in 32 bits");
    for (int i = 0; i < 3; i++) HIP_OR_FAIL(c, hipEventElapsedTime(&c->stage_ms[i], c->ev[i], c->ev[i + 1]));
    c->n_copy = n;
    c->n_sends = c->op == PCCL_OP_ALLREDUCE ? 2 * n : n;
    c->coll_time = c->op == PCCL_OP_ALLREDUCE ? 2 * h.cstar : h.cstar;
    c->have_result = true;
    c->have_receipts = false;
    if (n_sends) *n_sends = c->n_sends;
    if (collective_time_ns) *collective_time_ns = c->coll_time;
    return PCCL_OK;
}

pccl_status pccl_synthesize(pccl_ctx *c, uint64_t *n_sends, uint32_t *collective_time_ns)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    c->have_result = false;
    if (!c->have_ws) return fail(c, PCCL_ESTATE, "set a workspace first");
    return synthesize_bound(c, n_sends, collective_time_ns);
    GUARD_END(c)
}

pccl_status pccl_synthesize_static(pccl_ctx *c, uint64_t max_sends, void *hip_stream, uint64_t *n_sends,
                                   uint32_t *collective_time_ns)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    c->err.clear();
    c->have_result = false;
    if (!c->have_coll) return fail(c, PCCL_ESTATE, "set a collective first");
    if (!c->planned) return fail(c, PCCL_ESTATE, "the last pccl_set_collective / pccl_set_switch_model failed");
    void *base = g_scratch_ptr[c->device];
    if (!base) return fail(c, PCCL_EDEVICE, "no static scratch address for device %d", c->device);
    const uint64_t ms = max_sends ? max_sends : safe_max_sends(c);
    c->have_ws = false;
    pccl_status st = bind_workspace(c, static_cast<char *>(base), PCCL_STATIC_SCRATCH_BYTES, ms,
                                    static_cast<hipStream_t>(hip_stream), true);
    if (st != PCCL_OK) return st;
    {
        std::lock_guard<std::mutex> g(g_scratch_mu);
        ScratchOwner &o = g_scratch_owner[c->device];
        // the inputs are still there when this context (same plan and bound)
        // was the last to copy them in; otherwise they are copied again
        c->uploaded = o.serial == c->serial && o.plan_gen == c->plan_gen && o.max_sends == ms;
        o.serial = 0;
        c->static_call = ++o.call;
    }
    st = synthesize_bound(c, n_sends, collective_time_ns);
    {
        std::lock_guard<std::mutex> g(g_scratch_mu);
        ScratchOwner &o = g_scratch_owner[c->device];
        if (c->uploaded && o.call == c->static_call) {
            o.serial = c->serial;
            o.plan_gen = c->plan_gen;
            o.max_sends = ms;
        }
    }
    return st;
    GUARD_END(c)
}

pccl_status pccl_get_schedule(pccl_ctx *c, pccl_send *out, uint64_t capacity)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    if (capacity < c->n_sends) return fail(c, PCCL_EINVAL, "capacity %llu < %llu sends",
                                          (unsigned long long)capacity, (unsigned long long)c->n_sends);
    if (c->n_sends) {
        if (!out) return fail(c, PCCL_EINVAL, "null output");
        HIP_OR_FAIL(c, hipMemcpyAsync(out, c->ly.out, sizeof(pccl_send) * c->n_sends, hipMemcpyDefault, c->stream));
        HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
    }
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_get_path(pccl_ctx *c, uint32_t chunk, uint32_t device, uint32_t *t_start, uint32_t *next_device,
                          uint32_t capacity, uint32_t *length)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    if (chunk >= c->C) return fail(c, PCCL_EINVAL, "chunk %u out of range (%u chunks)", chunk, c->C);
    if (device >= c->D) return fail(c, PCCL_EINVAL, "device %u out of range (%u devices)", device, c->D);
    if (capacity && (!t_start || !next_device)) return fail(c, PCCL_EINVAL, "null output");
    if (!c->have_receipts) {
        // which transfer delivered each (chunk, device), from the copy schedule
        std::vector<pccl_send> s(c->n_sends);
        if (c->n_sends) {
            HIP_OR_FAIL(c, hipMemcpyAsync(s.data(), c->ly.out, sizeof(pccl_send) * c->n_sends, hipMemcpyDeviceToHost,
                                          c->stream));
            HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
        }
        const uint32_t cs = c->ctl_host.cstar;
        c->receipt.clear();
        c->receipt.reserve(c->n_copy * 2 + 1);
        for (const pccl_send &x : s) {
            uint32_t t = x.t_start_ns, l = x.link;
            if (c->op == PCCL_OP_REDUCE_REVERSED) {
                l = c->rev[x.link];
                t = cs - x.t_start_ns - c->T[l];
            } else if (c->op == PCCL_OP_ALLREDUCE) {
                if (x.flags & PCCL_SEND_REDUCE) continue;
                t -= cs;
            }
            c->receipt[((uint64_t)x.chunk << 32) | c->dst[l]] = ((uint64_t)l << 32) | t;
        }
        c->have_receipts = true;
    }
    // walk back from the device to the chunk's source
    std::vector<std::pair<uint32_t, uint32_t>> hops;
    uint32_t v = device;
    for (;;) {
        auto it = c->receipt.find(((uint64_t)chunk << 32) | v);
        if (it == c->receipt.end()) break;
        if (hops.size() >= c->D) return fail(c, PCCL_EINTERNAL, "delivery chain of chunk %u does not end", chunk);
        const uint32_t l = (uint32_t)(it->second >> 32);
        hops.emplace_back((uint32_t)it->second, v);
        v = c->src[l];
    }
    if (hops.empty()) return fail(c, PCCL_EINVAL, "device %u receives no copy of chunk %u", device, chunk);
    std::reverse(hops.begin(), hops.end());
    if (length) *length = (uint32_t)hops.size();
    for (uint32_t i = 0; i < hops.size() && i < capacity; i++) {
        t_start[i] = hops[i].first;
        next_device[i] = hops[i].second;
    }
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_export_program(pccl_ctx *c, pccl_step *steps, uint64_t step_capacity, uint32_t *deps,
                                uint64_t dep_capacity, uint64_t *n_steps, uint64_t *n_deps)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    std::vector<pccl_send> s(c->n_sends);
    if (c->n_sends) {
        HIP_OR_FAIL(c, hipMemcpyAsync(s.data(), c->ly.out, sizeof(pccl_send) * c->n_sends, hipMemcpyDeviceToHost,
                                      c->stream));
        HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
    }
    const uint32_t N = c->N;
    auto key = [](uint32_t chunk, uint32_t dev, uint32_t phase) {
        return ((uint64_t)phase << 63) | ((uint64_t)chunk << 32) | dev;
    };
    // a switch's copy came in over one transfer, and a partial sum leaves it
    // over one transfer; the All-Reduce's two halves are told apart by the
    // reduce flag
    std::unordered_map<uint64_t, uint64_t> into_sw, from_sw;
    for (uint64_t i = 0; i < s.size(); i++) {
        const uint32_t l = s[i].link, red = s[i].flags & PCCL_SEND_REDUCE;
        if (!red && c->dst[l] >= N) into_sw[key(s[i].chunk, c->dst[l], 0)] = i;
        if (red && c->src[l] >= N) from_sw[key(s[i].chunk, c->src[l], 1)] = i;
    }
    // NPU-to-NPU transfers with the switches folded away
    struct Xfer {
        uint32_t from, to, chunk, t, end, red;
    };
    std::vector<Xfer> xs;
    xs.reserve(s.size());
    for (const pccl_send &x : s) {
        const uint32_t l = x.link, red = x.flags & PCCL_SEND_REDUCE;
        if (!red) {
            if (c->dst[l] >= N) continue;  // carried on by the switch's out-transfers
            uint32_t u = c->src[l];
            for (uint32_t hop = 0; u >= N; hop++) {
                auto it = into_sw.find(key(x.chunk, u, 0));
                if (it == into_sw.end() || hop > c->D)
                    return fail(c, PCCL_EINTERNAL, "switch %u forwards chunk %u it never received", u, x.chunk);
                u = c->src[s[it->second].link];
            }
            xs.push_back({u, c->dst[l], x.chunk, x.t_start_ns, x.t_start_ns + c->T[l], 0u});
        } else {
            if (c->src[l] >= N) continue;  // folded into the transfers that fed the switch
            uint32_t v = c->dst[l], end = x.t_start_ns + c->T[l];
            for (uint32_t hop = 0; v >= N; hop++) {
                auto it = from_sw.find(key(x.chunk, v, 1));
                if (it == from_sw.end() || hop > c->D)
                    return fail(c, PCCL_EINTERNAL, "switch %u reduces chunk %u but never sends it on", v, x.chunk);
                const pccl_send &y = s[it->second];
                v = c->dst[y.link];
                end = y.t_start_ns + c->T[y.link];
            }
            xs.push_back({c->src[l], v, x.chunk, x.t_start_ns, end, 1u});
        }
    }
    // thread blocks: per rank, send blocks by ascending peer, then receive blocks
    std::vector<std::vector<uint32_t>> sendp(N), recvp(N);
    for (const Xfer &x : xs) {
        sendp[x.from].push_back(x.to);
        recvp[x.to].push_back(x.from);
    }
    for (uint32_t r = 0; r < N; r++) {
        for (auto *v : {&sendp[r], &recvp[r]}) {
            std::sort(v->begin(), v->end());
            v->erase(std::unique(v->begin(), v->end()), v->end());
        }
    }
    auto tb_of = [&](uint32_t r, uint32_t peer, bool send) {
        const auto &v = send ? sendp[r] : recvp[r];
        const uint32_t k = (uint32_t)(std::lower_bound(v.begin(), v.end(), peer) - v.begin());
        return send ? k : (uint32_t)sendp[r].size() + k;
    };
    struct Tmp {
        uint32_t rank, tb, op, peer, chunk, t, end;
    };
    std::vector<Tmp> st;
    st.reserve(2 * xs.size());
    for (const Xfer &x : xs) {
        st.push_back({x.from, tb_of(x.from, x.to, true), PCCL_STEP_SEND, x.to, x.chunk, x.t, x.end});
        st.push_back({x.to, tb_of(x.to, x.from, false), x.red ? PCCL_STEP_RECV_REDUCE : PCCL_STEP_RECV, x.from,
                      x.chunk, x.t, x.end});
    }
    std::sort(st.begin(), st.end(), [](const Tmp &a, const Tmp &b) {
        if (a.rank != b.rank) return a.rank < b.rank;
        if (a.tb != b.tb) return a.tb < b.tb;
        if (a.t != b.t) return a.t < b.t;
        return a.chunk < b.chunk;
    });
    // a send waits for the receives of its chunk on its rank that end before it starts
    std::unordered_map<uint64_t, std::vector<std::pair<uint32_t, uint32_t>>> recvs;  // (chunk, rank) -> (end, step)
    for (uint32_t i = 0; i < st.size(); i++)
        if (st[i].op != PCCL_STEP_SEND) recvs[key(st[i].chunk, st[i].rank, 0)].push_back({st[i].end, i});
    std::vector<uint32_t> dep_first(st.size(), 0), dep_count(st.size(), 0), dl;
    for (uint32_t i = 0; i < st.size(); i++) {
        dep_first[i] = (uint32_t)dl.size();
        if (st[i].op != PCCL_STEP_SEND) continue;
        auto it = recvs.find(key(st[i].chunk, st[i].rank, 0));
        if (it == recvs.end()) continue;
        for (const auto &e : it->second)
            if (e.first <= st[i].t) dl.push_back(e.second);
        dep_count[i] = (uint32_t)dl.size() - dep_first[i];
    }
    if (n_steps) *n_steps = st.size();
    if (n_deps) *n_deps = dl.size();
    if (!steps && !deps) return PCCL_OK;
    if (!steps || !deps || step_capacity < st.size() || dep_capacity < dl.size())
        return fail(c, PCCL_EINVAL, "program needs %zu steps and %zu dependencies", st.size(), dl.size());
    for (uint32_t i = 0; i < st.size(); i++)
        steps[i] = {st[i].rank, st[i].tb, st[i].op, st[i].peer, st[i].chunk, st[i].t, dep_first[i], dep_count[i]};
    if (!dl.empty()) std::memcpy(deps, dl.data(), sizeof(uint32_t) * dl.size());
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_get_matcher(pccl_ctx *c, uint32_t *kernel)
{
    if (!c || !kernel) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    *kernel = c->ran_sw ? 1u : 0u;
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_get_stats(pccl_ctx *c, uint64_t *events, uint64_t *rounds, uint64_t *clashes, uint64_t *windows)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    if (rounds) *rounds = c->ctl_host.rounds;
    if (clashes) *clashes = c->ctl_host.clashes;
    if (windows) *windows = c->ctl_host.windows;
    if (events) {
        // time 0 plus every distinct transfer end up to the last transfer start,
        // taken from the copy schedule
        std::vector<pccl_send> s(c->n_sends);
        if (c->n_sends) {
            HIP_OR_FAIL(c, hipMemcpyAsync(s.data(), c->ly.out, sizeof(pccl_send) * c->n_sends, hipMemcpyDeviceToHost,
                                          c->stream));
            HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
        }
        const uint32_t cs = c->ctl_host.cstar;
        std::vector<uint32_t> ends;
        ends.reserve(c->n_copy);
        uint32_t last = 0;
        for (const pccl_send &x : s) {
            uint32_t t = x.t_start_ns, l = x.link;
            if (c->op == PCCL_OP_REDUCE_REVERSED) {
                l = c->rev[x.link];
                t = cs - x.t_start_ns - c->T[l];
            } else if (c->op == PCCL_OP_ALLREDUCE) {
                if (x.flags & PCCL_SEND_REDUCE) continue;
                t -= cs;
            }
            last = std::max(last, t);
            ends.push_back(t + c->T[l]);
        }
        std::sort(ends.begin(), ends.end());
        ends.erase(std::unique(ends.begin(), ends.end()), ends.end());
        uint64_t e = 1;
        for (uint32_t x : ends)
            if (x <= last) e++;
        *events = e;
    }
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_get_link_usage(pccl_ctx *c, uint64_t *busy_ns, uint32_t n_bins, uint64_t *bin_busy_ns,
                                uint32_t *bin_ns)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c)) return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this schedule was reused" : "no schedule");
    if (bin_busy_ns && n_bins == 0) return fail(c, PCCL_EINVAL, "no bins");
    std::vector<pccl_send> s(c->n_sends);
    if (c->n_sends) {
        HIP_OR_FAIL(c, hipMemcpyAsync(s.data(), c->ly.out, sizeof(pccl_send) * c->n_sends, hipMemcpyDeviceToHost,
                                      c->stream));
        HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
    }
    if (busy_ns) {
        std::fill(busy_ns, busy_ns + c->L, 0ull);
        for (const pccl_send &x : s) busy_ns[x.link] += c->T[x.link];
    }
    if (bin_busy_ns) {
        const uint64_t ct = c->coll_time, w = std::max<uint64_t>(1, (ct + n_bins - 1) / n_bins);
        std::fill(bin_busy_ns, bin_busy_ns + n_bins, 0ull);
        for (const pccl_send &x : s) {
            const uint64_t a = x.t_start_ns, e = a + c->T[x.link];
            for (uint64_t b = a / w; b < n_bins && b * w < e; b++)
                bin_busy_ns[b] += std::min(e, (b + 1) * w) - std::max(a, b * w);
        }
        if (bin_ns) *bin_ns = (uint32_t)w;
    }
    return PCCL_OK;
    GUARD_END(c)
}

pccl_status pccl_get_profile(pccl_ctx *c, double *setup_ms, double *match_ms, double *output_ms,
                             uint64_t *scan_words)
{
    if (!c) return PCCL_EINVAL;
    if (!c->have_result) return fail(c, PCCL_ESTATE, "no synthesis");
    if (setup_ms) *setup_ms = c->stage_ms[0];
    if (match_ms) *match_ms = c->stage_ms[1];
    if (output_ms) *output_ms = c->stage_ms[2];
    if (scan_words) *scan_words = c->ctl_host.scan_words;
    return PCCL_OK;
}

pccl_status pccl_get_setup(pccl_ctx *c, uint32_t *link_time_ns, uint32_t *chunk_src, uint64_t *chunk_dist,
                           uint32_t *chunk_rank)
{
    if (!c) return PCCL_EINVAL;
    GUARD_BEGIN
    if (!result_alive(c))
        return fail(c, PCCL_ESTATE, c->have_result ? "the static scratch holding this synthesis was reused" : "no synthesis");
    if (link_time_ns && c->L) std::memcpy(link_time_ns, c->T.data(), sizeof(uint32_t) * c->L);
    hipStream_t st = c->stream;
    if (chunk_src && c->C)
        HIP_OR_FAIL(c, hipMemcpyAsync(chunk_src, c->ly.chunk_src, sizeof(uint32_t) * c->C, hipMemcpyDeviceToHost, st));
    if (chunk_dist && c->C)
        HIP_OR_FAIL(c, hipMemcpyAsync(chunk_dist, c->ly.chunk_dist, sizeof(uint64_t) * c->C, hipMemcpyDeviceToHost, st));
    if (chunk_rank && c->C)
        HIP_OR_FAIL(c, hipMemcpyAsync(chunk_rank, c->ly.rank, sizeof(uint32_t) * c->C, hipMemcpyDeviceToHost, st));
    HIP_OR_FAIL(c, hipStreamSynchronize(st));
    return PCCL_OK;
    GUARD_END(c)
}

}  // extern "C"
