// cb_api.cpp -- host side of the C ABI declared in include/cachebridge.h.
//
// Validation happens here, before anything is enqueued.  cb_plan_create turns
// the head map into the work items of the statistics kernel (CacheBridge
// Sec. 2.3: every map's support is known before fitting, so its reads are
// planned once) and into the source-block groups of the application kernel,
// and allocates the plan's workspace.  No other call allocates.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <functional>
#include <map>
#include <set>
#include <string>
#include <tuple>
#include <vector>

#include "cb_internal.h"

struct cb_plan {
    int device = 0;
    int n_cu = 256;
    int32_t n_maps = 0, L_s = 0, H_s = 0, d_s = 0, L_t = 0, H_t = 0, d_t = 0;
    int64_t max_tokens = 0;
    bool duplicate_targets = false;   // some target (layer, kv, head) has several maps (probes)
    // multi-layer feature (cb_plan_create_multi): k source layers per map
    bool multi = false;
    int32_t k = 1, P = 0, sample_stride = 1;
    int32_t n_tasks = 0;
    cb::MultiTask *d_tasks = nullptr;
    cb::ApplyMultiMap *d_amaps = nullptr;   // multi-layer application: map records, visiting order, layers
    int32_t *d_aorder = nullptr;
    int32_t *d_alayers = nullptr;
    int32_t *d_apairs = nullptr;            // multi-layer application: pair records (see ApplyMultiArgs)
    int32_t n_apairs = 0, apair_stride = 0;
    int32_t *d_asingles = nullptr;          // and the maps without a partner, in visiting order
    int32_t n_asingles = 0;
    int32_t *d_mwrow = nullptr;             // multi-layer: weight row of each map (means pass)
    // statistics schedule
    int32_t n_items = 0;
    int32_t max_chunks = 1;
    cb::StatsItem *d_items = nullptr;
    int32_t *d_map_item = nullptr;
    int32_t *d_map_slot = nullptr;
    int32_t *d_map_yown = nullptr;
    float *d_partials = nullptr;
    void *d_zero = nullptr;        // zero bytes: source of copies for absent tokens
    // application schedule and split coefficients
    int32_t n_groups = 0;
    cb::ApplyGroup *d_groups = nullptr;
    uint16_t *d_whi = nullptr;
    uint16_t *d_wlo = nullptr;
    float *d_bias = nullptr;
    // multi-layer plans with rotary keys: de-rotated K rows of the current call
    uint16_t *d_rws = nullptr;
    int64_t rws_bytes = 0;
};

namespace {

thread_local std::string g_last_error;

cb_status fail(cb_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

cb_status ok() {
    g_last_error.clear();
    return CB_OK;
}

bool supported_width(int d) { return d == 64 || d == 96 || d == 128; }

// Work units of a call: each item's token tiles (KT tokens of one sequence)
// are cut into n_chunks chunks of chunk_tiles tiles.  Enough (item, chunk)
// units to give every compute unit `per_cu` of them, at most 2048 tiles (64Ki
// tokens) per fp32 partial, and never more chunks than the plan's workspace
// holds (max_chunks <= 0: no such limit).
void choose_chunks(int64_t tiles, int n_items, int n_cu, int max_chunks, int *n_chunks, int *chunk_tiles,
                   int per_cu = 8) {
    if (tiles <= 0) {
        *n_chunks = 0;
        *chunk_tiles = 1;
        return;
    }
    const int64_t target_units = (int64_t)per_cu * n_cu;
    int64_t nc = (target_units + n_items - 1) / n_items;
    nc = std::max<int64_t>(nc, (tiles + 2047) / 2048);
    nc = std::min<int64_t>(nc, tiles);
    if (max_chunks > 0) nc = std::min<int64_t>(nc, max_chunks);
    nc = std::max<int64_t>(nc, 1);
    const int64_t ct = (tiles + nc - 1) / nc;
    *chunk_tiles = (int)ct;
    *n_chunks = (int)((tiles + ct - 1) / ct);
}

cb_status check_device(const cb_plan *p) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return fail(CB_ERR_DEVICE, "hipGetDevice failed");
    if (dev != p->device)
        return fail(CB_ERR_INVALID_ARGUMENT, "plan was created on device %d but device %d is current", p->device, dev);
    return CB_OK;
}

// Geometry and alignment of a cache used in a call.
cb_status check_cache(const char *name, const cb_cache *c, int L, int H, int d) {
    if (!c) return fail(CB_ERR_INVALID_ARGUMENT, "%s is NULL", name);
    if (c->n_layers != L || c->n_heads != H || c->head_dim != d)
        return fail(CB_ERR_SHAPE, "%s is %d layers x %d heads x %d, plan expects %d x %d x %d", name, c->n_layers,
                    c->n_heads, c->head_dim, L, H, d);
    if (c->n_seqs < 0 || c->seq_len < 0) return fail(CB_ERR_SHAPE, "%s has negative n_seqs or seq_len", name);
    if ((int64_t)c->n_seqs * c->seq_len > 0 && !c->data) return fail(CB_ERR_INVALID_ARGUMENT, "%s->data is NULL", name);
    const int64_t s[5] = {c->s_layer, c->s_kv, c->s_seq, c->s_head, c->s_tok};
    for (int i = 0; i < 5; ++i) {
        if (s[i] < 0) return fail(CB_ERR_SHAPE, "%s has a negative stride", name);
        if (s[i] % 8 != 0) return fail(CB_ERR_MISALIGNED, "%s strides must be multiples of 8 elements (16 bytes)", name);
    }
    if (((uintptr_t)c->data) % 16 != 0) return fail(CB_ERR_MISALIGNED, "%s->data is not 16-byte aligned", name);
    return CB_OK;
}

cb::Strides strides_of(const cb_cache *c) { return {c->s_layer, c->s_kv, c->s_seq, c->s_head, c->s_tok}; }

// Validation and work units shared by the statistics calls.  *empty is set
// for a call without tokens (nothing to enqueue).
cb_status prepare_stats(const cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                        int64_t w_row_stride, cb::StatsArgs &a, bool &empty) {
    if (cb_status s = check_cache("src", src, p->L_s, p->H_s, p->d_s)) return s;
    if (cb_status s = check_cache("tgt", tgt, p->L_t, p->H_t, p->d_t)) return s;
    if (src->n_seqs != tgt->n_seqs || src->seq_len != tgt->seq_len)
        return fail(CB_ERR_SHAPE, "src and tgt disagree on n_seqs / seq_len");
    const int64_t N = (int64_t)src->n_seqs * src->seq_len;
    if (N > p->max_tokens)
        return fail(CB_ERR_UNSUPPORTED, "call has %lld tokens, plan allows %lld", (long long)N, (long long)p->max_tokens);
    empty = N == 0;
    if (empty) return CB_OK;
    if (!weights) return fail(CB_ERR_INVALID_ARGUMENT, "weights is NULL");
    if (w_row_stride < N) return fail(CB_ERR_SHAPE, "w_row_stride (%lld) < tokens in the call (%lld)",
                                      (long long)w_row_stride, (long long)N);
    if (((uintptr_t)weights) % 4) return fail(CB_ERR_MISALIGNED, "weights must be 4-byte aligned");
    if (cb_status s = check_device(p)) return s;

    a.src = (const uint16_t *)src->data;
    a.tgt = (const uint16_t *)tgt->data;
    a.w = weights;
    a.ss = strides_of(src);
    a.ts = strides_of(tgt);
    a.w_row_stride = w_row_stride;
    const int64_t KT = cb::kStatsTileTokens;
    const int64_t tps = (src->seq_len + KT - 1) / KT;
    const int64_t tiles = (int64_t)src->n_seqs * tps;
    if (tiles > INT32_MAX) return fail(CB_ERR_UNSUPPORTED, "too many token tiles in one call");
    if (a.ss.tok * 2 * KT >= (1LL << 31) || a.ts.tok * 2 * KT >= (1LL << 31))
        return fail(CB_ERR_UNSUPPORTED, "token strides must be below 2^25 elements");
    a.seq_len = (uint32_t)src->seq_len;
    a.TPS = cb::make_fastdiv((uint32_t)tps);
    a.n_tiles = (int32_t)tiles;
    choose_chunks(tiles, p->n_items, p->n_cu, p->max_chunks, &a.n_chunks, &a.chunk_tiles);
    if (a.n_chunks > p->max_chunks) return fail(CB_ERR_UNSUPPORTED, "internal: chunk count exceeds workspace");
    a.n_items = p->n_items;
    a.items = p->d_items;
    a.partials = p->d_partials;
    a.zero = p->d_zero;
    return CB_OK;
}

// One task rectangle of a multi-layer map: row blocks {r0, r1} x column blocks
// {c0, c1} (block k is the target block, only ever c1), and the mask of the
// cells it keeps: bit 2 a + b is cell (row a, column b).
struct Rect { int r0, r1, c0, c1, mask; };

// Exact cover of the cells of a k-block map -- every unordered pair {i, j} of
// source blocks (i <= j) and every cell (i, target) -- by rectangles whose four
// cells are all needed and distinct, so no task computes a masked cell.  A
// depth-first search that always branches on the cell with the fewest
// remaining candidates; false when the cell count is not a multiple of four,
// for k above 16, or when no cover turns up within the node budget.  The
// result depends on k only.
bool exact_rect_cover(int k, std::vector<Rect> &out) {
    const int n_cells = k * (k + 1) / 2 + k;
    if (k < 2 || k > 16 || n_cells % 4 != 0) return false;
    const int Y = k;
    auto cell = [&](int a, int b) -> int {            // unordered source pair, or (a, target)
        if (b == Y) return k * (k + 1) / 2 + a;
        const int i = std::min(a, b), j = std::max(a, b);
        return i * k - i * (i - 1) / 2 + (j - i);
    };
    struct Cand { Rect r; int c[4]; };
    std::vector<Cand> cands;
    for (int r0 = 0; r0 < k; ++r0)
        for (int r1 = r0 + 1; r1 < k; ++r1)
            for (int c0 = 0; c0 < k; ++c0)
                for (int c1 = c0 + 1; c1 <= Y; ++c1) {
                    Cand x = {{r0, r1, c0, c1, 0xF}, {cell(r0, c0), cell(r0, c1), cell(r1, c0), cell(r1, c1)}};
                    bool distinct = true;
                    for (int a = 0; a < 4; ++a)
                        for (int b = a + 1; b < 4; ++b) distinct = distinct && x.c[a] != x.c[b];
                    if (distinct) cands.push_back(x);
                }
    std::vector<std::vector<int>> by_cell(n_cells);
    for (int i = 0; i < (int)cands.size(); ++i)
        for (int a = 0; a < 4; ++a) by_cell[cands[i].c[a]].push_back(i);
    std::vector<char> covered(n_cells, 0);
    std::vector<int> chosen;
    long nodes = 0;
    const long budget = 4000;
    auto fits = [&](int i) {
        for (int a = 0; a < 4; ++a)
            if (covered[cands[i].c[a]]) return false;
        return true;
    };
    std::function<bool(int)> rec = [&](int left) -> bool {
        if (left == 0) return true;
        if (++nodes > budget) return false;
        int best = -1, best_n = 1 << 30;
        for (int c = 0; c < n_cells; ++c) {
            if (covered[c]) continue;
            int cnt = 0;
            for (int i : by_cell[c]) cnt += fits(i);
            if (cnt < best_n) { best = c; best_n = cnt; }
            if (cnt == 0) return false;
        }
        for (int i : by_cell[best]) {
            if (!fits(i)) continue;
            for (int a = 0; a < 4; ++a) covered[cands[i].c[a]] = 1;
            chosen.push_back(i);
            if (rec(left - 4)) return true;
            chosen.pop_back();
            for (int a = 0; a < 4; ++a) covered[cands[i].c[a]] = 0;
        }
        return false;
    };
    if (!rec(n_cells)) return false;
    out.clear();
    for (int i : chosen) out.push_back(cands[i].r);
    return true;
}


// Validation and launch arguments of a multi-layer statistics call.
cb_status prepare_multi(const cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                        int64_t w_row_stride, cb::MultiArgs &a, bool &empty) {
    if (cb_status s = check_cache("src", src, p->L_s, p->H_s, p->d_s)) return s;
    if (cb_status s = check_cache("tgt", tgt, p->L_t, p->H_t, p->d_t)) return s;
    if (src->n_seqs != tgt->n_seqs || src->seq_len != tgt->seq_len)
        return fail(CB_ERR_SHAPE, "src and tgt disagree on n_seqs / seq_len");
    const int64_t N = (int64_t)src->n_seqs * src->seq_len;
    empty = N == 0;
    if (empty) return CB_OK;
    if (!weights) return fail(CB_ERR_INVALID_ARGUMENT, "weights is NULL");
    if (w_row_stride < N) return fail(CB_ERR_SHAPE, "w_row_stride (%lld) < tokens in the call (%lld)",
                                      (long long)w_row_stride, (long long)N);
    if (((uintptr_t)weights) % 4) return fail(CB_ERR_MISALIGNED, "weights must be 4-byte aligned");
    if (cb_status s = check_device(p)) return s;
    const int64_t KT = cb::kMultiTileRows;
    const int64_t rows = (src->seq_len + p->sample_stride - 1) / p->sample_stride;
    const int64_t tps = (rows + KT - 1) / KT;
    const int64_t tiles = (int64_t)src->n_seqs * tps;
    if (tiles > INT32_MAX - 16) return fail(CB_ERR_UNSUPPORTED, "too many row tiles in one call");
    const int64_t step = (int64_t)p->sample_stride * 2 * KT;
    if (src->s_tok * step >= (1LL << 31) || tgt->s_tok * step >= (1LL << 31))
        return fail(CB_ERR_UNSUPPORTED, "token stride x sample_stride too large (16 rows must span < 2 GiB)");
    a.src = (const uint16_t *)src->data;
    a.tgt = (const uint16_t *)tgt->data;
    a.w = weights;
    a.ss = strides_of(src);
    a.ts = strides_of(tgt);
    a.w_row_stride = w_row_stride;
    a.seq_len = (uint32_t)src->seq_len;
    a.stride = (uint32_t)p->sample_stride;
    a.rows_per_seq = (uint32_t)rows;
    a.TPS = cb::make_fastdiv((uint32_t)tps);
    a.n_tiles = (int32_t)tiles;
    {   // flush at most every kMultiFlushTiles tiles, at a multiple of six tiles (one loop trip)
        const int64_t iters = (tiles + 5) / 6 * 6;
        const int64_t nf = (iters + cb::kMultiFlushTiles - 1) / cb::kMultiFlushTiles;
        int64_t ct = (iters + nf - 1) / nf;
        ct = (ct + 5) / 6 * 6;
        a.chunk_tiles = (int32_t)ct;
    }
    a.n_tasks = p->n_tasks;
    a.per_xcd = (p->n_tasks + 7) / 8;
    a.k = p->k;
    a.P = p->P;
    a.d_t = p->d_t;
    a.tasks = p->d_tasks;
    a.zero = p->d_zero;
    return CB_OK;
}

cb::ReduceArgs reduce_args(const cb_plan *p, const cb::StatsArgs &a) {
    cb::ReduceArgs r = {};
    r.partials = p->d_partials;
    r.map_item = p->d_map_item;
    r.map_slot = p->d_map_slot;
    r.map_yown = p->d_map_yown;
    r.n_items = p->n_items;
    r.n_chunks = a.n_chunks;
    r.n_maps = p->n_maps;
    return r;
}

}  // namespace

extern "C" {

const char *cb_status_string(cb_status s) {
    switch (s) {
        case CB_OK: return "CB_OK";
        case CB_ERR_INVALID_ARGUMENT: return "CB_ERR_INVALID_ARGUMENT";
        case CB_ERR_SHAPE: return "CB_ERR_SHAPE";
        case CB_ERR_MISALIGNED: return "CB_ERR_MISALIGNED";
        case CB_ERR_OUT_OF_MEMORY: return "CB_ERR_OUT_OF_MEMORY";
        case CB_ERR_DEVICE: return "CB_ERR_DEVICE";
        case CB_ERR_UNSUPPORTED: return "CB_ERR_UNSUPPORTED";
    }
    return "CB_ERR_UNKNOWN";
}

const char *cb_last_error(void) { return g_last_error.c_str(); }

cb_status cb_plan_destroy(cb_plan *p) {
    if (!p) return ok();
    (void)hipDeviceSynchronize();
    (void)hipFree(p->d_items);
    (void)hipFree(p->d_map_item);
    (void)hipFree(p->d_map_slot);
    (void)hipFree(p->d_map_yown);
    (void)hipFree(p->d_partials);
    (void)hipFree(p->d_zero);
    (void)hipFree(p->d_groups);
    (void)hipFree(p->d_whi);
    (void)hipFree(p->d_wlo);
    (void)hipFree(p->d_bias);
    (void)hipFree(p->d_tasks);
    (void)hipFree(p->d_amaps);
    (void)hipFree(p->d_aorder);
    (void)hipFree(p->d_alayers);
    (void)hipFree(p->d_apairs);
    (void)hipFree(p->d_asingles);
    (void)hipFree(p->d_mwrow);
    (void)hipFree(p->d_rws);
    delete p;
    return ok();
}

cb_status cb_plan_create(const cb_head_map *map, const cb_cache *src_geom, const cb_cache *tgt_geom,
                         int64_t max_tokens_per_call, cb_plan **out) {
    if (!out) return fail(CB_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    if (!map || !src_geom || !tgt_geom) return fail(CB_ERR_INVALID_ARGUMENT, "map, src_geom and tgt_geom must be non-NULL");
    if (map->n_maps <= 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps must be positive (got %d)", map->n_maps);
    if (!map->tgt_layer || !map->tgt_head || !map->kv || !map->src_layer || !map->src_head || !map->weight_row)
        return fail(CB_ERR_INVALID_ARGUMENT, "every head map array must be non-NULL");
    const int L_s = src_geom->n_layers, H_s = src_geom->n_heads, d_s = src_geom->head_dim;
    const int L_t = tgt_geom->n_layers, H_t = tgt_geom->n_heads, d_t = tgt_geom->head_dim;
    if (L_s <= 0 || H_s <= 0 || L_t <= 0 || H_t <= 0)
        return fail(CB_ERR_SHAPE, "layer and head counts must be positive");
    if (!supported_width(d_s) || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "head widths must be 64, 96 or 128 (got d_s=%d, d_t=%d)", d_s, d_t);
    if (max_tokens_per_call < 0 || max_tokens_per_call > (int64_t)INT32_MAX - 65536)
        return fail(CB_ERR_UNSUPPORTED, "max_tokens_per_call must be in [0, 2^31 - 65537]");

    const int n = map->n_maps;
    std::set<std::tuple<int, int, int>> targets;
    bool duplicate = false;
    for (int m = 0; m < n; ++m) {
        const int tl = map->tgt_layer[m], th = map->tgt_head[m], z = map->kv[m];
        const int sl = map->src_layer[m], sh = map->src_head[m], wr = map->weight_row[m];
        if (tl < 0 || tl >= L_t || th < 0 || th >= H_t)
            return fail(CB_ERR_INVALID_ARGUMENT, "map %d: target (%d, %d) outside %d x %d", m, tl, th, L_t, H_t);
        if (sl < 0 || sl >= L_s || sh < 0 || sh >= H_s)
            return fail(CB_ERR_INVALID_ARGUMENT, "map %d: source (%d, %d) outside %d x %d", m, sl, sh, L_s, H_s);
        if (z != 0 && z != 1) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: kv must be 0 or 1 (got %d)", m, z);
        if (wr < 0) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: negative weight row", m);
        if (!targets.insert(std::make_tuple(tl, z, th)).second) duplicate = true;
    }

    cb_plan *p = new cb_plan();
    if (hipGetDevice(&p->device) != hipSuccess) {
        delete p;
        return fail(CB_ERR_DEVICE, "hipGetDevice failed (no HIP device?)");
    }
    int ncu = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, p->device) == hipSuccess && ncu > 0)
        p->n_cu = ncu;
    p->n_maps = n;
    p->L_s = L_s; p->H_s = H_s; p->d_s = d_s;
    p->L_t = L_t; p->H_t = H_t; p->d_t = d_t;
    p->max_tokens = max_tokens_per_call;
    p->duplicate_targets = duplicate;
    p->P = d_s + 1;

    // ---- group maps by source block, in order of first appearance
    std::map<std::tuple<int, int, int>, int> gid;
    std::vector<std::vector<int>> groups;
    for (int m = 0; m < n; ++m) {
        auto key = std::make_tuple(map->src_layer[m], map->kv[m], map->src_head[m]);
        auto it = gid.find(key);
        if (it == gid.end()) {
            gid.emplace(key, (int)groups.size());
            groups.push_back({m});
        } else {
            groups[it->second].push_back(m);
        }
    }

    // Target sums (sum w y, sum w y^2) depend only on the target block and the
    // weight row: the first map of each such pair carries them for all of its
    // maps, so the means pass reads every target row once per call.
    std::vector<int32_t> yown(n);
    {
        std::map<std::tuple<int, int, int, int>, int> first;
        for (int m = 0; m < n; ++m) {
            const auto key = std::make_tuple(map->tgt_layer[m], map->kv[m], map->tgt_head[m], map->weight_row[m]);
            auto f = first.find(key);
            if (f == first.end()) f = first.emplace(key, m).first;
            yown[m] = f->second;
        }
    }
    auto fill_slot = [&](cb::StatsItem &it, int s, int m) {
        it.map[s] = m;
        it.own_y[s] = yown[m] == m;
        it.src_layer[s] = map->src_layer[m];
        it.src_head[s] = map->src_head[m];
        it.kv[s] = map->kv[m];
        it.tgt_layer[s] = map->tgt_layer[m];
        it.tgt_head[s] = map->tgt_head[m];
        it.wrow[s] = map->weight_row[m];
    };
    std::vector<cb::StatsItem> items;
    std::vector<int> singles;
    for (const auto &g : groups) {
        size_t i = 0;
        for (; i + 1 < g.size(); i += 2) {
            cb::StatsItem it = {};
            it.n_slots = 2;
            it.shared_x = 1;
            fill_slot(it, 0, g[i]);
            fill_slot(it, 1, g[i + 1]);
            items.push_back(it);
        }
        if (i < g.size()) singles.push_back(g[i]);
    }
    for (size_t i = 0; i < singles.size(); i += 2) {
        cb::StatsItem it = {};
        fill_slot(it, 0, singles[i]);
        if (i + 1 < singles.size()) {
            it.n_slots = 2;
            fill_slot(it, 1, singles[i + 1]);
        } else {
            it.n_slots = 1;
            fill_slot(it, 1, singles[i]);   // unused slot mirrors slot 0 (never read)
        }
        it.shared_x = 0;
        items.push_back(it);
    }
    p->n_items = (int)items.size();
    std::vector<int32_t> map_item(n), map_slot(n);
    for (int i = 0; i < p->n_items; ++i)
        for (int s = 0; s < items[i].n_slots; ++s) {
            map_item[items[i].map[s]] = i;
            map_slot[items[i].map[s]] = s;
        }
    int nc = 1, ct = 1;
    const int64_t KT = cb::kStatsTileTokens;
    choose_chunks((std::max<int64_t>(max_tokens_per_call, 1) + KT - 1) / KT, p->n_items, p->n_cu, 0, &nc, &ct);
    p->max_chunks = std::max(nc, 1);

    std::vector<cb::ApplyGroup> agroups;
    for (const auto &g : groups) {
        for (size_t i = 0; i < g.size(); i += 2) {
            cb::ApplyGroup ag = {};
            ag.n_slots = (i + 1 < g.size()) ? 2 : 1;
            ag.src_layer = map->src_layer[g[i]];
            ag.src_head = map->src_head[g[i]];
            ag.kv = map->kv[g[i]];
            for (int s = 0; s < 2; ++s) {
                const int m = g[std::min(i + s, g.size() - 1)];
                ag.map[s] = m;
                ag.tgt_layer[s] = map->tgt_layer[m];
                ag.tgt_head[s] = map->tgt_head[m];
            }
            agroups.push_back(ag);
        }
    }
    p->n_groups = (int)agroups.size();

    // ---- device allocations
    const int64_t slot_floats = cb::stats_slot_floats(d_s, d_t);
    const size_t partial_bytes = (size_t)p->n_items * p->max_chunks * 2 * slot_floats * sizeof(float);
    const size_t wsplit = (size_t)n * d_t * d_s * sizeof(uint16_t);
    bool okm = hipMalloc(&p->d_items, sizeof(cb::StatsItem) * items.size()) == hipSuccess &&
               hipMalloc(&p->d_map_item, sizeof(int32_t) * n) == hipSuccess &&
               hipMalloc(&p->d_map_slot, sizeof(int32_t) * n) == hipSuccess &&
               hipMalloc(&p->d_map_yown, sizeof(int32_t) * n) == hipSuccess &&
               hipMalloc(&p->d_partials, partial_bytes) == hipSuccess &&
               hipMalloc(&p->d_zero, 256) == hipSuccess &&
               hipMalloc(&p->d_groups, sizeof(cb::ApplyGroup) * agroups.size()) == hipSuccess &&
               hipMalloc(&p->d_whi, wsplit) == hipSuccess && hipMalloc(&p->d_wlo, wsplit) == hipSuccess &&
               hipMalloc(&p->d_bias, sizeof(float) * n * d_t) == hipSuccess;
    if (!okm) {
        (void)hipGetLastError();
        cb_plan_destroy(p);
        return fail(CB_ERR_OUT_OF_MEMORY, "plan workspace allocation failed (%zu bytes of partial sums)", partial_bytes);
    }
    bool okc = hipMemset(p->d_zero, 0, 256) == hipSuccess &&
               hipMemcpy(p->d_items, items.data(), sizeof(cb::StatsItem) * items.size(), hipMemcpyHostToDevice) == hipSuccess &&
               hipMemcpy(p->d_map_item, map_item.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice) == hipSuccess &&
               hipMemcpy(p->d_map_slot, map_slot.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice) == hipSuccess &&
               hipMemcpy(p->d_map_yown, yown.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice) == hipSuccess &&
               hipMemcpy(p->d_groups, agroups.data(), sizeof(cb::ApplyGroup) * agroups.size(), hipMemcpyHostToDevice) == hipSuccess;
    if (!okc) {
        cb_plan_destroy(p);
        return fail(CB_ERR_DEVICE, "copying the schedule to the device failed");
    }
    *out = p;
    return ok();
}

// Pairs of maps for the multi-layer application: two maps of one (kv, source
// head) whose source-layer sets are equal (as multisets) share every staged
// block.  Maps are taken in visiting order (kv, source head, target layer,
// target head); within a run of one (kv, source head) the maps of each layer
// set pair up in that order, and an odd one out stays single.  Record of a
// pair (stride 4 + 3k): [0] map A, [1] map B, [2], [3] unused, [4 + j] the
// j-th layer of the set in ascending order, [4 + k + j] and [4 + 2k + j] A's
// and B's block index of that layer.
static std::vector<int32_t> build_pairs(const cb_head_map_multi *map, int n, int k, const std::vector<int> &order,
                                        int32_t *n_pairs, std::vector<int32_t> *singles) {
    const int stride = 4 + 3 * k;
    std::vector<int32_t> rec;
    auto sorted_blocks = [&](int m) {
        std::vector<std::pair<int32_t, int32_t>> v(k);       // (layer, block index)
        for (int i = 0; i < k; ++i) v[i] = {map->src_layers[(int64_t)m * k + i], i};
        std::stable_sort(v.begin(), v.end());
        return v;
    };
    int32_t np = 0;
    singles->clear();
    for (int g0 = 0; g0 < n;) {
        int g1 = g0 + 1;
        while (g1 < n && map->kv[order[g1]] == map->kv[order[g0]] &&
               map->src_head[order[g1]] == map->src_head[order[g0]])
            ++g1;
        std::map<std::vector<int32_t>, int> waiting;          // layer set -> a map still without partner
        std::vector<std::pair<int, int>> pr;                  // in the order the second member is met
        for (int i = g0; i < g1; ++i) {
            const int m = order[i];
            std::vector<int32_t> key;
            for (const auto &e : sorted_blocks(m)) key.push_back(e.first);
            auto it = waiting.find(key);
            if (it == waiting.end()) {
                waiting[key] = m;
            } else {
                pr.push_back({it->second, m});
                waiting.erase(it);
            }
        }
        for (const auto &ab : pr) {
            const auto A = sorted_blocks(ab.first), B = sorted_blocks(ab.second);
            std::vector<int32_t> r(stride, 0);
            r[0] = ab.first;
            r[1] = ab.second;
            for (int j = 0; j < k; ++j) {
                r[4 + j] = A[j].first;
                r[4 + k + j] = A[j].second;
                r[4 + 2 * k + j] = B[j].second;
            }
            rec.insert(rec.end(), r.begin(), r.end());
            ++np;
        }
        for (int i = g0; i < g1; ++i) {                       // the maps left alone, in visiting order
            const int m = order[i];
            for (const auto &w : waiting)
                if (w.second == m) singles->push_back(m);
        }
        g0 = g1;
    }
    *n_pairs = np;
    return rec;
}

cb_status cb_plan_create_multi(const cb_head_map_multi *map, const cb_cache *src_geom, const cb_cache *tgt_geom,
                               int32_t sample_stride, cb_plan **out) {
    if (!out) return fail(CB_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    if (!map || !src_geom || !tgt_geom) return fail(CB_ERR_INVALID_ARGUMENT, "map, src_geom and tgt_geom must be non-NULL");
    if (map->n_maps <= 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps must be positive (got %d)", map->n_maps);
    if (map->k < 1 || map->k > 32) return fail(CB_ERR_UNSUPPORTED, "k must be in 1..32 (got %d)", map->k);
    if (!map->tgt_layer || !map->tgt_head || !map->kv || !map->src_layers || !map->src_head || !map->weight_row)
        return fail(CB_ERR_INVALID_ARGUMENT, "every head map array must be non-NULL");
    if (sample_stride < 1) return fail(CB_ERR_INVALID_ARGUMENT, "sample_stride must be >= 1 (got %d)", sample_stride);
    const int L_s = src_geom->n_layers, H_s = src_geom->n_heads, d_s = src_geom->head_dim;
    const int L_t = tgt_geom->n_layers, H_t = tgt_geom->n_heads, d_t = tgt_geom->head_dim;
    if (L_s <= 0 || H_s <= 0 || L_t <= 0 || H_t <= 0) return fail(CB_ERR_SHAPE, "layer and head counts must be positive");
    if (d_s != 128 || d_t != 128)
        return fail(CB_ERR_UNSUPPORTED, "multi-layer maps need d_s = d_t = 128 (got d_s=%d, d_t=%d)", d_s, d_t);
    const int n = map->n_maps, k = map->k;
    std::set<std::tuple<int, int, int>> targets;
    bool duplicate = false;
    for (int m = 0; m < n; ++m) {
        const int tl = map->tgt_layer[m], th = map->tgt_head[m], z = map->kv[m];
        const int sh = map->src_head[m], wr = map->weight_row[m];
        if (tl < 0 || tl >= L_t || th < 0 || th >= H_t)
            return fail(CB_ERR_INVALID_ARGUMENT, "map %d: target (%d, %d) outside %d x %d", m, tl, th, L_t, H_t);
        if (sh < 0 || sh >= H_s) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: source head %d outside %d", m, sh, H_s);
        if (z != 0 && z != 1) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: kv must be 0 or 1 (got %d)", m, z);
        if (wr < 0) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: negative weight row", m);
        std::set<int> seen;
        for (int i = 0; i < k; ++i) {
            const int sl = map->src_layers[(int64_t)m * k + i];
            if (sl < 0 || sl >= L_s) return fail(CB_ERR_INVALID_ARGUMENT, "map %d: source layer %d outside %d", m, sl, L_s);
            if (!seen.insert(sl).second)
                return fail(CB_ERR_INVALID_ARGUMENT, "map %d: source layer %d selected twice", m, sl);
        }
        if (!targets.insert(std::make_tuple(tl, z, th)).second) duplicate = true;
    }

    cb_plan *p = new cb_plan();
    if (hipGetDevice(&p->device) != hipSuccess) {
        delete p;
        return fail(CB_ERR_DEVICE, "hipGetDevice failed (no HIP device?)");
    }
    int ncu = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, p->device) == hipSuccess && ncu > 0)
        p->n_cu = ncu;
    p->n_maps = n;
    p->L_s = L_s; p->H_s = H_s; p->d_s = d_s;
    p->L_t = L_t; p->H_t = H_t; p->d_t = d_t;
    p->max_tokens = INT64_MAX;
    p->duplicate_targets = duplicate;
    p->multi = true;
    p->k = k;
    p->P = k * d_s + 1;
    p->sample_stride = sample_stride;

    // ---- statistics tasks.  Maps are visited by (kv, source head, target
    // layer, target head): neighbouring maps then read mostly the same source
    // blocks, and the kernel hands each XCD a contiguous run of tasks.  The
    // cells of a map (every unordered pair {i, j} of source blocks, the k
    // diagonal blocks and the k (i, target) cells) are packed into equal
    // rectangles {r0, r1} x {c0, c1}; a pair may be computed in either
    // orientation because G is mirrored:
    //   couple (a, b) = (2m, 2m+1):   {a, b} x {a, y}   -> (a,a) {a,b} (a,y) (b,y)
    //   couples m < m':               {a, b} x {a', b'} -> four pairs
    //   the diagonals (b, b) left by the couples, two at a time:
    //                                 {b, b'} x {b, b'} -> (b,b) (b',b') (the pair is already done)
    //   an unpaired last block c:     {c, c} x {c, y}, then its pairs with
    //                                 the couples, {c, c} x {a, b} (half used)
    // That gives 12 tasks for the 44 cells of k = 8.  When the cell count is a
    // multiple of four, an exact cover by full rectangles is searched first
    // (exact_rect_cover); at k = 8 it has 11 tasks and no unused cell.
    std::vector<int> order(n);
    for (int m = 0; m < n; ++m) order[m] = m;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
        return std::make_tuple(map->kv[a], map->src_head[a], map->tgt_layer[a], map->tgt_head[a]) <
               std::make_tuple(map->kv[b], map->src_head[b], map->tgt_layer[b], map->tgt_head[b]);
    });
    std::vector<Rect> rects;
    const int Y = k;
    const int nc = k / 2;
    if (exact_rect_cover(k, rects)) {
        // every rectangle does four needed cells (k = 8: 11 tasks instead of 12)
    } else {
    for (int m = 0; m < nc; ++m) rects.push_back({2 * m, 2 * m + 1, 2 * m, Y, 0xF});
    for (int m = 0; m < nc; ++m)
        for (int m2 = m + 1; m2 < nc; ++m2) rects.push_back({2 * m, 2 * m + 1, 2 * m2, 2 * m2 + 1, 0xF});
    for (int m = 0; m < nc; m += 2) {
        const int b = 2 * m + 1;
        if (m + 1 < nc) {
            const int b2 = 2 * m + 3;
            rects.push_back({b, b2, b, b2, 0x9});            // cells (b, b) and (b2, b2)
        } else {
            rects.push_back({b, b, b, b, 0x1});              // a lone leftover diagonal
        }
    }
    if (k % 2) {
        const int c = k - 1;
        rects.push_back({c, c, c, Y, 0x3});                  // (c, c) and (c, y)
        for (int m = 0; m < nc; ++m) rects.push_back({c, c, 2 * m, 2 * m + 1, 0x3});
    }
    }
    std::vector<cb::MultiTask> tasks;
    for (int m : order) {
        const int32_t *S = map->src_layers + (int64_t)m * k;
        std::vector<char> own_x(k, 0);
        bool own_w = false, own_y = false;
        for (const Rect &rc : rects) {
            cb::MultiTask t = {};
            t.map = m;
            t.wrow = map->weight_row[m];
            t.kv = map->kv[m];
            t.tgt_layer = map->tgt_layer[m];
            t.tgt_head = map->tgt_head[m];
            t.src_head = map->src_head[m];
            t.rows[0] = rc.r0; t.rows[1] = rc.r1;
            t.cols[0] = rc.c0; t.cols[1] = rc.c1;
            t.cell_mask = rc.mask;
            int blk[4];
            t.n_lds = 0;
            auto slot_of = [&](int b) {
                for (int s2 = 0; s2 < t.n_lds; ++s2)
                    if (blk[s2] == b) return s2;
                blk[t.n_lds] = b;
                t.slot_layer[t.n_lds] = b < k ? S[b] : -1;
                return t.n_lds++;
            };
            t.row_slot[0] = slot_of(rc.r0);
            t.row_slot[1] = slot_of(rc.r1);
            t.col_slot[0] = slot_of(rc.c0);
            t.col_slot[1] = slot_of(rc.c1);
            for (int s2 = t.n_lds; s2 < 4; ++s2) t.slot_layer[s2] = t.slot_layer[0];
            for (int a2 = 0; a2 < 2; ++a2) {
                const int r = a2 == 0 ? rc.r0 : rc.r1;
                const bool used = ((rc.mask >> (2 * a2)) & 3) != 0;
                if (used && !own_x[r] && !(a2 == 1 && rc.r1 == rc.r0)) {
                    own_x[r] = 1;
                    t.flags |= 1 << a2;
                }
            }
            if (!own_w && (t.flags & 1) && rc.r0 == 0) {
                own_w = true;
                t.flags |= 4;
            }
            if (!own_y && rc.c1 == Y) {
                own_y = true;
                t.flags |= 8;
            }
            tasks.push_back(t);
        }
    }
    p->n_tasks = (int32_t)tasks.size();
    std::vector<int32_t> singles;
    const std::vector<int32_t> pairs = build_pairs(map, n, k, order, &p->n_apairs, &singles);
    p->apair_stride = 4 + 3 * k;
    p->n_asingles = (int32_t)singles.size();

    std::vector<cb::ApplyMultiMap> amaps(n);
    for (int m = 0; m < n; ++m) amaps[m] = {map->tgt_layer[m], map->tgt_head[m], map->kv[m], map->src_head[m]};
    const size_t wsplit = (size_t)n * d_t * (size_t)(k * d_s) * sizeof(uint16_t);
    bool okm = hipMalloc(&p->d_tasks, sizeof(cb::MultiTask) * tasks.size()) == hipSuccess &&
               hipMalloc(&p->d_zero, 256) == hipSuccess &&
               hipMalloc(&p->d_amaps, sizeof(cb::ApplyMultiMap) * n) == hipSuccess &&
               hipMalloc(&p->d_aorder, sizeof(int32_t) * n) == hipSuccess &&
               hipMalloc(&p->d_alayers, sizeof(int32_t) * (size_t)n * k) == hipSuccess &&
               hipMalloc(&p->d_apairs, sizeof(int32_t) * (pairs.size() + 1)) == hipSuccess &&
               hipMalloc(&p->d_asingles, sizeof(int32_t) * (singles.size() + 1)) == hipSuccess &&
               hipMalloc(&p->d_mwrow, sizeof(int32_t) * (size_t)n) == hipSuccess &&
               hipMalloc(&p->d_whi, 2 * wsplit) == hipSuccess &&   // hi and lo fragment planes
               hipMalloc(&p->d_bias, sizeof(float) * n * d_t) == hipSuccess;
    if (!okm) {
        (void)hipGetLastError();
        cb_plan_destroy(p);
        return fail(CB_ERR_OUT_OF_MEMORY, "plan allocation failed");
    }
    if (hipMemset(p->d_zero, 0, 256) != hipSuccess ||
        hipMemcpy(p->d_tasks, tasks.data(), sizeof(cb::MultiTask) * tasks.size(), hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(p->d_amaps, amaps.data(), sizeof(cb::ApplyMultiMap) * n, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(p->d_aorder, order.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice) != hipSuccess ||
        hipMemcpy(p->d_alayers, map->src_layers, sizeof(int32_t) * (size_t)n * k, hipMemcpyHostToDevice) != hipSuccess ||
        (!pairs.empty() &&
         hipMemcpy(p->d_apairs, pairs.data(), sizeof(int32_t) * pairs.size(), hipMemcpyHostToDevice) != hipSuccess) ||
        (!singles.empty() &&
         hipMemcpy(p->d_asingles, singles.data(), sizeof(int32_t) * singles.size(), hipMemcpyHostToDevice) != hipSuccess) ||
        hipMemcpy(p->d_mwrow, map->weight_row, sizeof(int32_t) * (size_t)n, hipMemcpyHostToDevice) != hipSuccess) {
        cb_plan_destroy(p);
        return fail(CB_ERR_DEVICE, "copying the schedule to the device failed");
    }
    *out = p;
    return ok();
}

cb_status cb_plan_feature_width(const cb_plan *p, int32_t *P, int32_t *k) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (P) *P = p->P;
    if (k) *k = p->k;
    return ok();
}

cb_status cb_plan_shape(const cb_plan *p, int32_t *n_maps, int32_t *d_s, int32_t *d_t) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (n_maps) *n_maps = p->n_maps;
    if (d_s) *d_s = p->d_s;
    if (d_t) *d_t = p->d_t;
    return ok();
}

cb_status cb_stats_zero(const cb_plan *p, float *G, float *C, void *stream) {
    if (!p || !G || !C) return fail(CB_ERR_INVALID_ARGUMENT, "plan, G and C must be non-NULL");
    if (cb_status s = check_device(p)) return s;
    const int64_t P = p->P;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_fill_zero(G, (int64_t)p->n_maps * P * P, st) != hipSuccess ||
        cb::launch_fill_zero(C, (int64_t)p->n_maps * P * p->d_t, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "fill kernel launch failed");
    return ok();
}

// A rotary spec against the head width it turns and the positions a call needs.
static cb_status check_rope(const char *name, const cb_rope_spec *r, int32_t head_dim, int64_t seq_len) {
    if (!r->table) return fail(CB_ERR_INVALID_ARGUMENT, "%s->table is NULL", name);
    if (r->style != CB_ROPE_HALF_SPLIT && r->style != CB_ROPE_INTERLEAVED)
        return fail(CB_ERR_INVALID_ARGUMENT, "%s: unknown rope style %d", name, r->style);
    if (r->head_dim != head_dim)
        return fail(CB_ERR_SHAPE, "%s was built for head_dim %d, the cache it turns has %d", name, r->head_dim,
                    head_dim);
    if (r->pos_offset < 0 || (int64_t)r->pos_offset + seq_len > (int64_t)r->n_pos)
        return fail(CB_ERR_SHAPE, "%s: positions %d .. %lld need a table of that many rows (n_pos = %d)", name,
                    r->pos_offset, (long long)r->pos_offset + seq_len - 1, r->n_pos);
    if (((uintptr_t)r->table) % 16) return fail(CB_ERR_MISALIGNED, "%s->table must be 16-byte aligned", name);
    return CB_OK;
}

cb_status cb_stats_accumulate(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                              int64_t w_row_stride, float *G, float *C, void *stream) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!G || !C) return fail(CB_ERR_INVALID_ARGUMENT, "G and C must be non-NULL");
    if (((uintptr_t)G) % 4 || ((uintptr_t)C) % 4) return fail(CB_ERR_MISALIGNED, "G and C must be 4-byte aligned");
    if (p->multi) {
        cb::MultiArgs ma = {};
        bool empty = false;
        if (cb_status s = prepare_multi(p, src, tgt, weights, w_row_stride, ma, empty)) return s;
        if (empty) return ok();
        ma.G = G;
        ma.C = C;
        if (cb::launch_stats_multi(ma, (hipStream_t)stream) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer statistics kernel launch failed");
        return ok();
    }
    cb::StatsArgs a = {};
    bool empty = false;
    if (cb_status s = prepare_stats(p, src, tgt, weights, w_row_stride, a, empty)) return s;
    if (empty) return ok();
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_stats(p->d_s, p->d_t, a, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "statistics kernel launch failed");
    cb::ReduceArgs r = reduce_args(p, a);
    r.G = G;
    r.C = C;
    if (cb::launch_reduce(p->d_s, p->d_t, r, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "reduction kernel launch failed");
    return ok();
}

// The rotation workspace of a multi-layer plan, grown to `bytes` (the old one
// is released once the device has finished with it).
static cb_status ensure_rws(cb_plan *p, int64_t bytes) {
    if (bytes <= p->rws_bytes) return CB_OK;
    (void)hipDeviceSynchronize();
    (void)hipFree(p->d_rws);
    p->d_rws = nullptr;
    p->rws_bytes = 0;
    if (hipMalloc((void **)&p->d_rws, (size_t)bytes) != hipSuccess)
        return fail(CB_ERR_OUT_OF_MEMORY, "rotation workspace of %lld bytes", (long long)bytes);
    p->rws_bytes = bytes;
    return CB_OK;
}

// The K rows of cache c at tokens 0, stride, 2 stride, ... turned back by
// their positions' angles (cb_rope's inverse arithmetic) into dst, compact:
// [layer][seq][head][row][d] with rows = ceil(seq_len / stride); its strides
// go to *view (kv unused).
static cb_status derotate_rows(const cb_cache *c, const cb_rope_spec *r, int32_t stride, uint16_t *dst,
                               cb::Strides *view, hipStream_t st) {
    const int64_t rows = (c->seq_len + stride - 1) / stride;
    const int64_t d = c->head_dim;
    view->tok = d;
    view->head = rows * d;
    view->seq = (int64_t)c->n_heads * rows * d;
    view->layer = (int64_t)c->n_seqs * view->seq;
    view->kv = 0;
    cb::RopeLaunch L = {};
    L.in = (const uint16_t *)c->data;
    L.out = dst;
    L.is = strides_of(c);
    L.is.tok = c->s_tok * stride;
    L.os = *view;
    L.table = r->table;
    L.n_layers = c->n_layers;
    L.n_heads = c->n_heads;
    L.n_seqs = c->n_seqs;
    L.seq_len = (int32_t)rows;
    L.d = (int32_t)d;
    L.style = r->style;
    L.pos_offset = r->pos_offset;
    L.pos_step = stride;
    L.inverse = 1;
    L.copy_v = 0;                                        // K rows only
    if (cb::launch_rope(L, st) != hipSuccess) return fail(CB_ERR_DEVICE, "rope launch failed");
    return CB_OK;
}

// Multi-layer statistics with rotary keys: each calibration row of a K block
// is staged by many tasks (every task of every map that reads the block), so
// the calibration rows are turned back once, gathered into a compact
// workspace, and the K tasks read them from there.
static cb_status stats_multi_rope(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                                  int64_t w_row_stride, float *G, float *C, const cb_rope_spec *src_rope,
                                  const cb_rope_spec *tgt_rope, void *stream) {
    cb::MultiArgs ma = {};
    bool empty = false;
    if (cb_status s = prepare_multi(p, src, tgt, weights, w_row_stride, ma, empty)) return s;
    if (empty) return ok();
    const int64_t rows = ma.rows_per_seq;
    const int64_t sb = src_rope ? (int64_t)p->L_s * src->n_seqs * p->H_s * rows * p->d_s : 0;
    const int64_t tb = tgt_rope ? (int64_t)p->L_t * tgt->n_seqs * p->H_t * rows * p->d_t : 0;
    if (cb_status s = ensure_rws(p, 2 * (sb + tb))) return s;
    hipStream_t st = (hipStream_t)stream;
    if (src_rope) {
        if (cb_status s = derotate_rows(src, src_rope, p->sample_stride, p->d_rws, &ma.ssk, st)) return s;
        ma.srck = p->d_rws;
    }
    if (tgt_rope) {
        if (cb_status s = derotate_rows(tgt, tgt_rope, p->sample_stride, p->d_rws + sb, &ma.tsk, st)) return s;
        ma.tgtk = p->d_rws + sb;
    }
    ma.G = G;
    ma.C = C;
    if (cb::launch_stats_multi(ma, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "multi-layer statistics kernel launch failed");
    return ok();
}

cb_status cb_stats_accumulate_rope(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                                   int64_t w_row_stride, float *G, float *C, const cb_rope_spec *src_rope,
                                   const cb_rope_spec *tgt_rope, void *stream) {
    if (!src_rope && !tgt_rope) return cb_stats_accumulate(p, src, tgt, weights, w_row_stride, G, C, stream);
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!G || !C) return fail(CB_ERR_INVALID_ARGUMENT, "G and C must be non-NULL");
    if (((uintptr_t)G) % 4 || ((uintptr_t)C) % 4) return fail(CB_ERR_MISALIGNED, "G and C must be 4-byte aligned");
    if (!src || !tgt) return fail(CB_ERR_INVALID_ARGUMENT, "src and tgt must be non-NULL");
    if (src_rope)
        if (cb_status s = check_rope("src_rope", src_rope, p->d_s, src->seq_len)) return s;
    if (tgt_rope)
        if (cb_status s = check_rope("tgt_rope", tgt_rope, p->d_t, tgt->seq_len)) return s;
    if (p->multi) return stats_multi_rope(p, src, tgt, weights, w_row_stride, G, C, src_rope, tgt_rope, stream);
    if (p->d_s != p->d_t || (p->d_s != 64 && p->d_s != 128))
        return fail(CB_ERR_UNSUPPORTED, "the fused de-rotation takes d_s = d_t = 64 or 128 (got %d, %d); "
                                        "turn the caches with cb_rope first", p->d_s, p->d_t);
    if (src_rope && tgt_rope && src_rope->style != tgt_rope->style)
        return fail(CB_ERR_UNSUPPORTED, "the fused de-rotation takes one pairing style for both caches");
    cb::StatsArgs a = {};
    bool empty = false;
    if (cb_status s = prepare_stats(p, src, tgt, weights, w_row_stride, a, empty)) return s;
    if (empty) return ok();
    const cb_rope_spec *r0 = src_rope ? src_rope : tgt_rope, *r1 = tgt_rope ? tgt_rope : src_rope;
    a.rope_tab[0] = r0->table;
    a.rope_tab[1] = r1->table;
    a.rope_pos[0] = r0->pos_offset;
    a.rope_pos[1] = r1->pos_offset;
    a.rope_on[0] = src_rope != nullptr;
    a.rope_on[1] = tgt_rope != nullptr;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_stats_rope(p->d_s, r0->style, a, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "statistics kernel launch failed");
    cb::ReduceArgs r = reduce_args(p, a);
    r.G = G;
    r.C = C;
    if (cb::launch_reduce(p->d_s, p->d_t, r, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "reduction kernel launch failed");
    return ok();
}

cb_status cb_stats_zero_centered(const cb_plan *p, double *sums, double *sq, float *A, float *B, void *stream) {
    if (!p || !sums || !A || !B) return fail(CB_ERR_INVALID_ARGUMENT, "plan, sums, A and B must be non-NULL");
    if (p->multi && sq) return fail(CB_ERR_UNSUPPORTED, "sums of squares (probes) are single-layer only");
    if (cb_status s = check_device(p)) return s;
    const int64_t n = p->n_maps, ds = p->multi ? (int64_t)p->P - 1 : p->d_s, dt = p->d_t;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_fill_zero((float *)sums, 2 * n * (1 + ds + dt), st) != hipSuccess ||
        (sq && cb::launch_fill_zero((float *)sq, 2 * n * (ds + dt), st) != hipSuccess) ||
        cb::launch_fill_zero(A, n * ds * ds, st) != hipSuccess || cb::launch_fill_zero(B, n * ds * dt, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "fill kernel launch failed");
    return ok();
}

// Pass-1 arguments of a multi-layer call (tgt_only: sum w and sum w y alone).
static cb::MeansMultiArgs means_multi_args(const cb_plan *p, const cb_cache *src, const cb::MultiArgs &ma,
                                           double *sums, bool tgt_only) {
    cb::MeansMultiArgs m = {};
    m.src = ma.src;
    m.tgt = ma.tgt;
    m.w = ma.w;
    m.ss = ma.ss;
    m.ts = ma.ts;
    m.w_row_stride = ma.w_row_stride;
    m.n_seqs = src->n_seqs;
    m.seq_len = src->seq_len;
    m.stride = p->sample_stride;
    m.rows_per_seq = (int32_t)ma.rows_per_seq;
    m.n_maps = p->n_maps;
    m.k = p->k;
    m.d_t = p->d_t;
    m.maps = p->d_amaps;
    m.layers = p->d_alayers;
    m.wrow = p->d_mwrow;
    m.sums = sums;
    m.tgt_only = tgt_only ? 1 : 0;
    return m;
}

cb_status cb_stats_means(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                         int64_t w_row_stride, double *sums, double *sq, void *stream) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!sums) return fail(CB_ERR_INVALID_ARGUMENT, "sums must be non-NULL");
    if (((uintptr_t)sums) % 8 || ((uintptr_t)sq) % 8) return fail(CB_ERR_MISALIGNED, "sums and sq must be 8-byte aligned");
    if (p->multi) {
        if (sq) return fail(CB_ERR_UNSUPPORTED, "sums of squares (probes) are single-layer only");
        cb::MultiArgs ma = {};
        bool empty = false;
        if (cb_status s = prepare_multi(p, src, tgt, weights, w_row_stride, ma, empty)) return s;
        if (empty) return ok();
        const cb::MeansMultiArgs m = means_multi_args(p, src, ma, sums, false);
        if (cb::launch_means_multi(m, (hipStream_t)stream) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer means kernel launch failed");
        return ok();
    }
    cb::StatsArgs a = {};
    bool empty = false;
    if (cb_status s = prepare_stats(p, src, tgt, weights, w_row_stride, a, empty)) return s;
    if (empty) return ok();
    hipStream_t st = (hipStream_t)stream;
    // The means partials are small ([unit][2][entries] fp64), so pass 1 cuts
    // the tiles finer than the moments pass, within the same workspace.
    {
        const int64_t ne = 1 + p->d_s + p->d_t + (sq ? p->d_s + p->d_t : 0);
        const int64_t cap = (int64_t)p->max_chunks * cb::stats_slot_floats(p->d_s, p->d_t) / (2 * ne);
        choose_chunks(a.n_tiles, p->n_items, p->n_cu, (int)std::min<int64_t>(cap, 1 << 20), &a.n_chunks,
                      &a.chunk_tiles, 16);
    }
    if (cb::launch_means(p->d_s, p->d_t, a, sq != nullptr, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "means kernel launch failed");
    cb::ReduceArgs r = reduce_args(p, a);
    r.sums = sums;
    r.sq = sq;
    if (cb::launch_means_reduce(p->d_s, p->d_t, r, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "means reduction launch failed");
    return ok();
}

cb_status cb_stats_accumulate_centered(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                                       int64_t w_row_stride, const double *sums, float *A, float *B, void *stream) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!sums || !A || !B) return fail(CB_ERR_INVALID_ARGUMENT, "sums, A and B must be non-NULL");
    if (((uintptr_t)sums) % 8 || ((uintptr_t)A) % 4 || ((uintptr_t)B) % 4)
        return fail(CB_ERR_MISALIGNED, "sums must be 8-byte and A, B 4-byte aligned");
    if (p->multi) {
        cb::MultiArgs ma = {};
        bool empty = false;
        if (cb_status s = prepare_multi(p, src, tgt, weights, w_row_stride, ma, empty)) return s;
        if (empty) return ok();
        ma.G = A;
        ma.C = B;
        ma.sums = sums;
        if (cb::launch_stats_multi_centered(ma, (hipStream_t)stream) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer centered statistics kernel launch failed");
        return ok();
    }
    cb::StatsArgs a = {};
    bool empty = false;
    if (cb_status s = prepare_stats(p, src, tgt, weights, w_row_stride, a, empty)) return s;
    if (empty) return ok();
    a.sums = sums;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_stats_centered(p->d_s, p->d_t, a, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "centered statistics kernel launch failed");
    cb::ReduceArgs r = reduce_args(p, a);
    r.G = A;
    r.C = B;
    r.sums = const_cast<double *>(sums);      // read only by the centered reduction
    if (cb::launch_reduce_centered(p->d_s, p->d_t, r, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "centered reduction launch failed");
    return ok();
}

cb_status cb_stats_accumulate_shifted(cb_plan *p, const cb_cache *src, const cb_cache *tgt, const float *weights,
                                      int64_t w_row_stride, const double *shift, double *sums, float *A, float *B,
                                      void *stream) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!shift || !sums || !A || !B) return fail(CB_ERR_INVALID_ARGUMENT, "shift, sums, A and B must be non-NULL");
    if (((uintptr_t)shift) % 8 || ((uintptr_t)sums) % 8 || ((uintptr_t)A) % 4 || ((uintptr_t)B) % 4)
        return fail(CB_ERR_MISALIGNED, "shift and sums must be 8-byte and A, B 4-byte aligned");
    if (shift == sums) return fail(CB_ERR_INVALID_ARGUMENT, "shift and sums must be different arrays");
    if (p->multi) {
        cb::MultiArgs ma = {};
        bool empty = false;
        if (cb_status s = prepare_multi(p, src, tgt, weights, w_row_stride, ma, empty)) return s;
        if (empty) return ok();
        ma.G = A;
        ma.C = B;
        ma.sums = shift;
        ma.resid = sums;
        // the moments and sum w (x - mu') here; sum w and sum w y from the target rows alone
        const cb::MeansMultiArgs m = means_multi_args(p, src, ma, sums, true);
        if (cb::launch_stats_multi_centered(ma, (hipStream_t)stream) != hipSuccess ||
            cb::launch_means_multi(m, (hipStream_t)stream) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer centered statistics kernel launch failed");
        return ok();
    }
    cb::StatsArgs a = {};
    bool empty = false;
    if (cb_status s = prepare_stats(p, src, tgt, weights, w_row_stride, a, empty)) return s;
    if (empty) return ok();
    a.sums = shift;
    a.bias_sums = 1;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_stats_centered(p->d_s, p->d_t, a, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "centered statistics kernel launch failed");
    cb::ReduceArgs r = reduce_args(p, a);
    r.G = A;
    r.C = B;
    r.sums = const_cast<double *>(shift);     // read only by the centered reduction
    r.resid = sums;
    if (cb::launch_reduce_centered(p->d_s, p->d_t, r, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "centered reduction launch failed");
    return ok();
}

cb_status cb_stats_shift_finish(const cb_plan *p, const double *shift, double *sums, float *A, float *B, void *stream) {
    if (!p || !shift || !sums || !A || !B)
        return fail(CB_ERR_INVALID_ARGUMENT, "plan, shift, sums, A and B must be non-NULL");
    if (((uintptr_t)shift) % 8 || ((uintptr_t)sums) % 8 || ((uintptr_t)A) % 4 || ((uintptr_t)B) % 4)
        return fail(CB_ERR_MISALIGNED, "shift and sums must be 8-byte and A, B 4-byte aligned");
    if (shift == sums) return fail(CB_ERR_INVALID_ARGUMENT, "shift and sums must be different arrays");
    if (cb_status s = check_device(p)) return s;
    const int32_t dx = p->multi ? p->P - 1 : p->d_s;
    if (cb::launch_shift_finish(p->n_maps, dx, p->d_t, shift, sums, A, B, (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "shift finish launch failed");
    return ok();
}

cb_status cb_ridge_solve(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                         uint32_t flags, float *maps, int32_t *info, void *stream) {
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (P > 129 && supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "P = %d: systems wider than 129 are solved by cb_ridge_solve_ws", P);
    if (!supported_width(P - 1) || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "P must be 65, 97 or 129 and d_t 64, 96 or 128 (got P=%d, d_t=%d)", P, d_t);
    if (flags & ~(uint32_t)(CB_LAMBDA_RELATIVE | CB_RIDGE_BIAS_UNPENALIZED))
        return fail(CB_ERR_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    if (!std::isfinite(lambda) || lambda < 0.f) return fail(CB_ERR_INVALID_ARGUMENT, "lambda must be finite and >= 0");
    if (n_maps == 0) return ok();
    if (!G || !C || !maps || !info) return fail(CB_ERR_INVALID_ARGUMENT, "G, C, maps and info must be non-NULL");
    if (((uintptr_t)G) % 4 || ((uintptr_t)C) % 4 || ((uintptr_t)maps) % 4 || ((uintptr_t)info) % 4)
        return fail(CB_ERR_MISALIGNED, "G, C, maps and info must be 4-byte aligned");
    if (cb::launch_solve(n_maps, P, d_t, G, C, lambda, flags, maps, info, (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "ridge solve launch failed");
    return ok();
}

int64_t cb_ridge_solve_workspace_bytes(int32_t P, int32_t d_t, int32_t n_systems) {
    if (P <= 129 || d_t < 1 || n_systems < 1) return 0;
    return cb::solve_blocked_bytes_per_system(P, d_t) * (int64_t)n_systems;
}

cb_status cb_ridge_solve_ws(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                            uint32_t flags, void *workspace, int64_t workspace_bytes, float *maps, int32_t *info,
                            void *stream) {
    if (P <= 129) return cb_ridge_solve(n_maps, P, d_t, G, C, lambda, flags, maps, info, stream);
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (P > 4097 || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "need P <= 4097 and d_t in {64, 96, 128} (got P=%d, d_t=%d)", P, d_t);
    if (flags & ~(uint32_t)(CB_LAMBDA_RELATIVE | CB_RIDGE_BIAS_UNPENALIZED))
        return fail(CB_ERR_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    if (!std::isfinite(lambda) || lambda < 0.f) return fail(CB_ERR_INVALID_ARGUMENT, "lambda must be finite and >= 0");
    if (n_maps == 0) return ok();
    if (!G || !C || !maps || !info || !workspace)
        return fail(CB_ERR_INVALID_ARGUMENT, "G, C, maps, info and workspace must be non-NULL");
    if (((uintptr_t)G) % 4 || ((uintptr_t)C) % 4 || ((uintptr_t)maps) % 4 || ((uintptr_t)info) % 4 ||
        ((uintptr_t)workspace) % 8)
        return fail(CB_ERR_MISALIGNED, "G, C, maps, info must be 4-byte and workspace 8-byte aligned");
    const int64_t need = cb::solve_blocked_bytes_per_system(P, d_t);
    if (workspace_bytes < need)
        return fail(CB_ERR_SHAPE, "workspace of %lld bytes is below one system's %lld bytes", (long long)workspace_bytes,
                    (long long)need);
    if (cb::launch_solve_blocked(n_maps, P, d_t, G, C, lambda, flags, workspace, workspace_bytes, maps, info,
                                 (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "blocked ridge solve launch failed");
    return ok();
}

cb_status cb_ridge_solve_noalloc(int32_t n_maps, int32_t P, int32_t d_t, const float *G, const float *C, float lambda,
                                 uint32_t flags, float *maps, int32_t *info, void *stream) {
    if (P <= 129) return cb_ridge_solve(n_maps, P, d_t, G, C, lambda, flags, maps, info, stream);
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (P > 4097 || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "need P <= 4097 and d_t in {64, 96, 128} (got P=%d, d_t=%d)", P, d_t);
    const int64_t need = cb::solve_blocked_bytes_per_system(P, d_t);
    if (need > cb::kStaticSolveScratchBytes)
        return fail(CB_ERR_UNSUPPORTED,
                    "one system of P=%d, d_t=%d needs %lld bytes of scratch; the allocation-free solve holds %lld "
                    "(use cb_ridge_solve_ws)",
                    P, d_t, (long long)need, (long long)cb::kStaticSolveScratchBytes);
    if (flags & ~(uint32_t)(CB_LAMBDA_RELATIVE | CB_RIDGE_BIAS_UNPENALIZED))
        return fail(CB_ERR_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    if (!std::isfinite(lambda) || lambda < 0.f) return fail(CB_ERR_INVALID_ARGUMENT, "lambda must be finite and >= 0");
    if (n_maps == 0) return ok();
    if (!G || !C || !maps || !info) return fail(CB_ERR_INVALID_ARGUMENT, "G, C, maps and info must be non-NULL");
    if (((uintptr_t)G) % 4 || ((uintptr_t)C) % 4 || ((uintptr_t)maps) % 4 || ((uintptr_t)info) % 4)
        return fail(CB_ERR_MISALIGNED, "G, C, maps and info must be 4-byte aligned");
    if (cb::launch_solve_blocked_static(n_maps, P, d_t, G, C, lambda, flags, maps, info, (hipStream_t)stream) !=
        hipSuccess)
        return fail(CB_ERR_DEVICE, "allocation-free blocked ridge solve failed (scratch lookup or launch)");
    return ok();
}

int64_t cb_ridge_solve_noalloc_max_bytes(void) { return cb::kStaticSolveScratchBytes; }

cb_status cb_ridge_solve_centered(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const float *A,
                                  const float *B, float lambda, uint32_t flags, float *maps, int32_t *info,
                                  void *stream) {
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (!supported_width(d_s) || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "d_s and d_t must be 64, 96 or 128 (got d_s=%d, d_t=%d)", d_s, d_t);
    if (flags & ~(uint32_t)(CB_LAMBDA_RELATIVE | CB_RIDGE_BIAS_UNPENALIZED))
        return fail(CB_ERR_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    if (!std::isfinite(lambda) || lambda < 0.f) return fail(CB_ERR_INVALID_ARGUMENT, "lambda must be finite and >= 0");
    if (n_maps == 0) return ok();
    if (!sums || !A || !B || !maps || !info)
        return fail(CB_ERR_INVALID_ARGUMENT, "sums, A, B, maps and info must be non-NULL");
    if (((uintptr_t)sums) % 8 || ((uintptr_t)A) % 4 || ((uintptr_t)B) % 4 || ((uintptr_t)maps) % 4 ||
        ((uintptr_t)info) % 4)
        return fail(CB_ERR_MISALIGNED, "sums must be 8-byte and A, B, maps, info 4-byte aligned");
    if (cb::launch_solve_centered(n_maps, d_s, d_t, sums, A, B, lambda, flags, maps, info, (hipStream_t)stream) !=
        hipSuccess)
        return fail(CB_ERR_DEVICE, "centered ridge solve launch failed");
    return ok();
}

cb_status cb_ridge_solve_centered_ws(int32_t n_maps, int32_t d_x, int32_t d_t, const double *sums, const float *A,
                                     const float *B, float lambda, uint32_t flags, void *workspace,
                                     int64_t workspace_bytes, float *maps, int32_t *info, void *stream) {
    if (d_x <= 128) return cb_ridge_solve_centered(n_maps, d_x, d_t, sums, A, B, lambda, flags, maps, info, stream);
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (d_x > 4096 || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "need d_x <= 4096 and d_t in {64, 96, 128} (got d_x=%d, d_t=%d)", d_x, d_t);
    if (flags & ~(uint32_t)(CB_LAMBDA_RELATIVE | CB_RIDGE_BIAS_UNPENALIZED))
        return fail(CB_ERR_INVALID_ARGUMENT, "unknown flag bits 0x%x", flags);
    if (!std::isfinite(lambda) || lambda < 0.f) return fail(CB_ERR_INVALID_ARGUMENT, "lambda must be finite and >= 0");
    if (n_maps == 0) return ok();
    if (!sums || !A || !B || !maps || !info || !workspace)
        return fail(CB_ERR_INVALID_ARGUMENT, "sums, A, B, maps, info and workspace must be non-NULL");
    if (((uintptr_t)sums) % 8 || ((uintptr_t)A) % 4 || ((uintptr_t)B) % 4 || ((uintptr_t)maps) % 4 ||
        ((uintptr_t)info) % 4 || ((uintptr_t)workspace) % 8)
        return fail(CB_ERR_MISALIGNED, "sums and workspace must be 8-byte and A, B, maps, info 4-byte aligned");
    const int64_t need = cb::solve_blocked_bytes_per_system(d_x, d_t);
    if (workspace_bytes < need)
        return fail(CB_ERR_SHAPE, "workspace of %lld bytes is below one system's %lld bytes", (long long)workspace_bytes,
                    (long long)need);
    if (cb::launch_solve_blocked(n_maps, d_x, d_t, A, B, lambda, flags, workspace, workspace_bytes, maps, info,
                                 (hipStream_t)stream, sums) != hipSuccess)
        return fail(CB_ERR_DEVICE, "blocked centered ridge solve launch failed");
    return ok();
}

cb_status cb_probe_r2(int32_t n_maps, int32_t d_s, int32_t d_t, const double *sums, const double *sq, const float *A,
                      const float *B, const float *maps, double *r2, void *stream) {
    if (n_maps < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_maps is negative");
    if (!supported_width(d_s) || !supported_width(d_t))
        return fail(CB_ERR_UNSUPPORTED, "d_s and d_t must be 64, 96 or 128 (got d_s=%d, d_t=%d)", d_s, d_t);
    if (n_maps == 0) return ok();
    if (!sums || !sq || !A || !B || !maps || !r2)
        return fail(CB_ERR_INVALID_ARGUMENT, "sums, sq, A, B, maps and r2 must be non-NULL");
    if (((uintptr_t)sums) % 8 || ((uintptr_t)sq) % 8 || ((uintptr_t)r2) % 8 || ((uintptr_t)A) % 4 ||
        ((uintptr_t)B) % 4 || ((uintptr_t)maps) % 4)
        return fail(CB_ERR_MISALIGNED, "sums, sq, r2 must be 8-byte and A, B, maps 4-byte aligned");
    if (cb::launch_probe_r2(n_maps, d_s, d_t, sums, sq, A, B, maps, r2, (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "probe R^2 launch failed");
    return ok();
}

cb_status cb_select_layers(const cb_head_map *map, const double *r2, int32_t n_tgt_layers, int32_t n_src_layers,
                           int32_t k, int32_t *selected, double *score) {
    if (!map || !r2 || !selected) return fail(CB_ERR_INVALID_ARGUMENT, "map, r2 and selected must be non-NULL");
    if (!map->tgt_layer || !map->src_layer) return fail(CB_ERR_INVALID_ARGUMENT, "map->tgt_layer and src_layer must be non-NULL");
    if (map->n_maps < 0 || n_tgt_layers <= 0 || n_src_layers <= 0 || k <= 0)
        return fail(CB_ERR_INVALID_ARGUMENT, "n_maps >= 0 and positive layer counts and k are required");
    const int64_t cells = (int64_t)n_tgt_layers * n_src_layers;
    std::vector<double> sum(cells, 0.0);
    std::vector<int64_t> cnt(cells, 0);
    for (int m = 0; m < map->n_maps; ++m) {
        const int l = map->tgt_layer[m], j = map->src_layer[m];
        if (l < 0 || l >= n_tgt_layers || j < 0 || j >= n_src_layers)
            return fail(CB_ERR_INVALID_ARGUMENT, "map %d: layer pair (%d, %d) outside %d x %d", m, l, j, n_tgt_layers,
                        n_src_layers);
        sum[(int64_t)l * n_src_layers + j] += r2[m];
        cnt[(int64_t)l * n_src_layers + j] += 1;
    }
    std::vector<int> order(n_src_layers);
    for (int l = 0; l < n_tgt_layers; ++l) {
        std::vector<double> sc(n_src_layers);
        for (int j = 0; j < n_src_layers; ++j) {
            const int64_t c = (int64_t)l * n_src_layers + j;
            sc[j] = cnt[c] ? sum[c] / (double)cnt[c] : -HUGE_VAL;
            if (score) score[c] = sc[j];
        }
        for (int j = 0; j < n_src_layers; ++j) order[j] = j;
        std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return sc[a] > sc[b]; });
        int n = 0;
        for (int j : order)
            if (n < k && cnt[(int64_t)l * n_src_layers + j]) selected[(int64_t)l * k + n++] = j;
        for (; n < k; ++n) selected[(int64_t)l * k + n] = -1;
    }
    return ok();
}

cb_status cb_attn_sensitivity(const cb_cache *tgt, const cb_queries *q, const int32_t *boundaries,
                              int32_t sample_stride, float *r, int64_t r_row_stride, void *stream) {
    if (!tgt || !q || !boundaries || !r) return fail(CB_ERR_INVALID_ARGUMENT, "tgt, q, boundaries and r must be non-NULL");
    const int d = tgt->head_dim;
    if (d != 64 && d != 128) return fail(CB_ERR_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", d);
    if (tgt->n_layers <= 0 || tgt->n_heads <= 0) return fail(CB_ERR_SHAPE, "tgt needs positive layer and head counts");
    if (cb_status s = check_cache("tgt", tgt, tgt->n_layers, tgt->n_heads, d)) return s;
    if (q->n_layers != tgt->n_layers || q->n_seqs != tgt->n_seqs || q->head_dim != d)
        return fail(CB_ERR_SHAPE, "q is %d layers x %d seqs x %d, tgt %d x %d x %d", q->n_layers, q->n_seqs, q->head_dim,
                    tgt->n_layers, tgt->n_seqs, d);
    if (q->n_qheads <= 0 || q->n_qheads % tgt->n_heads != 0)
        return fail(CB_ERR_SHAPE, "n_qheads (%d) must be a positive multiple of n_heads (%d)", q->n_qheads, tgt->n_heads);
    const int G = q->n_qheads / tgt->n_heads;
    if (G > 32 || (G & (G - 1)) != 0) return fail(CB_ERR_UNSUPPORTED, "query heads per KV head must be a power of two <= 32");
    const int nb = q->n_bounds;
    if (nb < 1 || nb > 64 || nb * G > 256)
        return fail(CB_ERR_UNSUPPORTED, "need 1 <= n_bounds <= 64 and n_bounds * G <= 256 (got %d, G = %d)", nb, G);
    if (sample_stride < 1) return fail(CB_ERR_INVALID_ARGUMENT, "sample_stride must be >= 1");
    for (int k = 0; k < nb; ++k) {
        if (boundaries[k] < 0 || boundaries[k] >= tgt->seq_len || (k > 0 && boundaries[k] <= boundaries[k - 1]))
            return fail(CB_ERR_INVALID_ARGUMENT, "boundaries must increase strictly within [0, seq_len)");
    }
    const int64_t N = (int64_t)tgt->n_seqs * tgt->seq_len;
    if (r_row_stride < N) return fail(CB_ERR_SHAPE, "r_row_stride (%lld) < tokens in the call (%lld)", (long long)r_row_stride,
                                      (long long)N);
    if (N == 0) return ok();
    if (!q->data) return fail(CB_ERR_INVALID_ARGUMENT, "q->data is NULL");
    const int64_t qs[4] = {q->s_layer, q->s_seq, q->s_bnd, q->s_head};
    for (int i = 0; i < 4; ++i)
        if (qs[i] < 0 || qs[i] % 8) return fail(CB_ERR_MISALIGNED, "q strides must be non-negative multiples of 8 elements");
    if (((uintptr_t)q->data) % 16 || ((uintptr_t)r) % 4) return fail(CB_ERR_MISALIGNED, "q->data must be 16-byte and r 4-byte aligned");
    if ((int64_t)tgt->n_seqs * tgt->n_layers * tgt->n_heads > INT32_MAX)
        return fail(CB_ERR_UNSUPPORTED, "too many (sequence, layer, head) units in one call");
    cb::AttnLaunch L = {};
    L.kv = (const uint16_t *)tgt->data;
    L.ts = strides_of(tgt);
    L.q = (const uint16_t *)q->data;
    for (int i = 0; i < 4; ++i) L.q_strides[i] = qs[i];
    L.n_layers = tgt->n_layers;
    L.n_heads = tgt->n_heads;
    L.G = G;
    L.n_bounds = nb;
    L.seq_len = tgt->seq_len;
    L.n_seqs = tgt->n_seqs;
    L.stride = sample_stride;
    L.d = d;
    L.bounds = boundaries;
    L.r = r;
    L.r_row_stride = r_row_stride;
    if (cb::launch_attn_sensitivity(L, (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "attention sensitivity launch failed");
    return ok();
}

cb_status cb_attn_weights(int32_t n_rows, int32_t n_seqs, int32_t seq_len, int32_t sample_stride, const float *r,
                          int64_t r_row_stride, int32_t p, float *w, int64_t w_row_stride, float *alpha,
                          void *stream) {
    if (n_rows < 0 || n_seqs < 0 || seq_len < 0) return fail(CB_ERR_INVALID_ARGUMENT, "negative size");
    if (sample_stride < 1 || p < 1) return fail(CB_ERR_INVALID_ARGUMENT, "sample_stride and p must be >= 1");
    const int64_t N = (int64_t)n_seqs * seq_len;
    if (r_row_stride < N || w_row_stride < N) return fail(CB_ERR_SHAPE, "row strides must be >= n_seqs * seq_len");
    if (n_rows == 0) return ok();
    if (!r || !w || !alpha) return fail(CB_ERR_INVALID_ARGUMENT, "r, w and alpha must be non-NULL");
    if (((uintptr_t)r) % 4 || ((uintptr_t)w) % 4 || ((uintptr_t)alpha) % 4)
        return fail(CB_ERR_MISALIGNED, "r, w and alpha must be 4-byte aligned");
    if (cb::launch_attn_weights(n_rows, n_seqs, seq_len, sample_stride, r, r_row_stride, p, w, w_row_stride, alpha,
                                (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "attention weights launch failed");
    return ok();
}

cb_status cb_rope_table(double theta, int32_t head_dim, int32_t n_pos, float *table, void *stream) {
    if (!(theta > 0.0) || !std::isfinite(theta)) return fail(CB_ERR_INVALID_ARGUMENT, "theta must be finite and > 0");
    if (head_dim < 2 || head_dim > 256 || head_dim % 2) return fail(CB_ERR_UNSUPPORTED, "head_dim must be even, 2..256");
    if (n_pos < 0) return fail(CB_ERR_INVALID_ARGUMENT, "n_pos is negative");
    if (n_pos == 0) return ok();
    if (!table) return fail(CB_ERR_INVALID_ARGUMENT, "table is NULL");
    if (((uintptr_t)table) % 8) return fail(CB_ERR_MISALIGNED, "table must be 8-byte aligned");
    if (cb::launch_rope_table(head_dim, n_pos, theta, table, (hipStream_t)stream) != hipSuccess)
        return fail(CB_ERR_DEVICE, "rope table launch failed");
    return ok();
}

cb_status cb_rope(const cb_cache *in, const cb_cache *out, const cb_rope_spec *rope, int32_t inverse, void *stream) {
    if (!in || !out || !rope) return fail(CB_ERR_INVALID_ARGUMENT, "in, out and rope must be non-NULL");
    const int d = in->head_dim;
    if (d < 16 || d > 256 || d % 16) return fail(CB_ERR_UNSUPPORTED, "head_dim must be a multiple of 16 up to 256");
    if (in->n_layers <= 0 || in->n_heads <= 0) return fail(CB_ERR_SHAPE, "in needs positive layer and head counts");
    if (cb_status s = check_cache("in", in, in->n_layers, in->n_heads, d)) return s;
    if (cb_status s = check_cache("out", out, in->n_layers, in->n_heads, d)) return s;
    if (out->n_seqs != in->n_seqs || out->seq_len != in->seq_len)
        return fail(CB_ERR_SHAPE, "in and out disagree on n_seqs / seq_len");
    if (cb_status s = check_rope("rope", rope, d, in->seq_len)) return s;
    if ((int64_t)in->n_seqs * in->seq_len == 0) return ok();
    const float *table = rope->table;
    const int32_t style = rope->style, pos_offset = rope->pos_offset;
    const bool same = in->data == out->data;
    if (same && (in->s_layer != out->s_layer || in->s_kv != out->s_kv || in->s_seq != out->s_seq ||
                 in->s_head != out->s_head || in->s_tok != out->s_tok))
        return fail(CB_ERR_INVALID_ARGUMENT, "an in-place transform needs out to have in's strides");
    cb::RopeLaunch L = {};
    L.in = (const uint16_t *)in->data;
    L.out = (uint16_t *)out->data;
    L.is = strides_of(in);
    L.os = strides_of(out);
    L.table = table;
    L.n_layers = in->n_layers;
    L.n_heads = in->n_heads;
    L.n_seqs = in->n_seqs;
    L.seq_len = in->seq_len;
    L.d = d;
    L.style = style;
    L.pos_offset = pos_offset;
    L.inverse = inverse ? 1 : 0;
    L.copy_v = same ? 0 : 1;
    L.pos_step = 1;
    if (cb::launch_rope(L, (hipStream_t)stream) != hipSuccess) return fail(CB_ERR_DEVICE, "rope launch failed");
    return ok();
}

// Single-layer application, optionally with the sender's rotary transform
// removed from the K source rows as they land (src_rope) and the target's
// applied to the K outputs before their rounding (tgt_rope); both specs are
// checked by the caller.
static cb_status apply_single(cb_plan *p, const float *maps, const cb_cache *src, const cb_cache *tgt_out,
                              const cb_rope_spec *src_rope, const cb_rope_spec *tgt_rope, void *stream) {
    if (p->duplicate_targets)
        return fail(CB_ERR_INVALID_ARGUMENT, "the plan maps some target (layer, kv, head) more than once; "
                                             "cb_apply needs one map per target");
    if (!maps) return fail(CB_ERR_INVALID_ARGUMENT, "maps is NULL");
    if (cb_status s = check_cache("src", src, p->L_s, p->H_s, p->d_s)) return s;
    if (cb_status s = check_cache("tgt_out", tgt_out, p->L_t, p->H_t, p->d_t)) return s;
    if (src->n_seqs != tgt_out->n_seqs || src->seq_len != tgt_out->seq_len)
        return fail(CB_ERR_SHAPE, "src and tgt_out disagree on n_seqs / seq_len");
    if (((uintptr_t)maps) % 4) return fail(CB_ERR_MISALIGNED, "maps must be 4-byte aligned");
    const int64_t N = (int64_t)src->n_seqs * src->seq_len;
    if (N > (int64_t)INT32_MAX - 4096) return fail(CB_ERR_UNSUPPORTED, "too many tokens in one call");
    if (src_rope && p->d_s != 64 && p->d_s != 128)
        return fail(CB_ERR_UNSUPPORTED, "the fused source de-rotation takes d_s = 64 or 128 (got %d); "
                                        "turn the sender with cb_rope first", p->d_s);
    if (cb_status s = check_device(p)) return s;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_split_maps(p->n_maps, p->d_s, p->d_t, maps, p->d_whi, p->d_wlo, p->d_bias, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "map split launch failed");
    if (N == 0) return ok();
    cb::ApplyArgs a = {};
    a.src = (const uint16_t *)src->data;
    a.out = (uint16_t *)tgt_out->data;
    a.ss = strides_of(src);
    a.os = strides_of(tgt_out);
    a.T = cb::make_fastdiv((uint32_t)src->seq_len);
    a.N = (int32_t)N;
    // Token tiles of whole 32-token sub-blocks: about 16 workgroups per
    // compute unit in total, at most 8192 tokens (a workgroup streams its
    // tile through a ring, so longer tiles amortize the ring's fill).
    {
        const int64_t target = 16LL * p->n_cu;
        int64_t tt = ((int64_t)N * std::max(p->n_groups, 1) + target - 1) / target;
        tt = std::min<int64_t>(std::max<int64_t>(tt, 256), 8192);
        tt = (tt + 31) / 32 * 32;
        a.tile_tokens = (int32_t)tt;
    }
    a.n_tiles = (int32_t)((N + a.tile_tokens - 1) / a.tile_tokens);
    a.groups = p->d_groups;
    a.w_hi = p->d_whi;
    a.w_lo = p->d_wlo;
    a.bias = p->d_bias;
    a.rope_table = tgt_rope ? tgt_rope->table : nullptr;
    a.rope_style = tgt_rope ? tgt_rope->style : 0;
    a.rope_pos_offset = tgt_rope ? tgt_rope->pos_offset : 0;
    a.src_rope_table = src_rope ? src_rope->table : nullptr;
    a.src_rope_style = src_rope ? src_rope->style : 0;
    a.src_rope_pos_offset = src_rope ? src_rope->pos_offset : 0;
    if ((int64_t)p->n_groups * a.n_tiles > (int64_t)INT32_MAX)
        return fail(CB_ERR_UNSUPPORTED, "too many application workgroups");
    if (cb::launch_apply(p->d_s, p->d_t, p->n_groups, a, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "application kernel launch failed");
    return ok();
}

// Multi-layer application, optionally with the sender's K rows turned back
// first (src_rope: one rotation pass into the plan's workspace, which the K
// maps then read; every source row is read by several maps) and the target's
// rotation fused into the epilogue (tgt_rope); both specs checked by the caller.
static cb_status apply_multi(cb_plan *p, const float *maps, const cb_cache *src, const cb_cache *tgt_out,
                             const cb_rope_spec *src_rope, const cb_rope_spec *tgt_rope, void *stream) {
    if (p->duplicate_targets)
        return fail(CB_ERR_INVALID_ARGUMENT, "the plan maps some target (layer, kv, head) more than once; "
                                             "cb_apply needs one map per target");
    if (!maps) return fail(CB_ERR_INVALID_ARGUMENT, "maps is NULL");
    if (cb_status s = check_cache("src", src, p->L_s, p->H_s, p->d_s)) return s;
    if (cb_status s = check_cache("tgt_out", tgt_out, p->L_t, p->H_t, p->d_t)) return s;
    if (src->n_seqs != tgt_out->n_seqs || src->seq_len != tgt_out->seq_len)
        return fail(CB_ERR_SHAPE, "src and tgt_out disagree on n_seqs / seq_len");
    if (((uintptr_t)maps) % 4) return fail(CB_ERR_MISALIGNED, "maps must be 4-byte aligned");
    const int64_t N = (int64_t)src->n_seqs * src->seq_len;
    if (N > (int64_t)INT32_MAX - 4096) return fail(CB_ERR_UNSUPPORTED, "too many tokens in one call");
    // the kernel addresses a row by a 32-bit byte offset from its (layer, kv, head) base
    if (N > 0 && 2 * ((int64_t)(src->n_seqs - 1) * src->s_seq + (int64_t)(src->seq_len - 1) * src->s_tok + 128) >
                     (int64_t)UINT32_MAX)
        return fail(CB_ERR_UNSUPPORTED, "src rows of one (layer, kv, head) span more than 4 GiB; "
                                        "apply in smaller batches");
    if (src_rope && N > 0 &&
        2 * ((int64_t)(src->n_seqs - 1) * p->H_s * src->seq_len * p->d_s + (int64_t)src->seq_len * p->d_s) >
            (int64_t)UINT32_MAX)
        return fail(CB_ERR_UNSUPPORTED, "the de-rotated rows of one (layer, head) would span more than 4 GiB; "
                                        "apply in smaller batches");
    if (cb_status s = check_device(p)) return s;
    hipStream_t st = (hipStream_t)stream;
    if (cb::launch_split_maps_frag(p->n_maps, p->k, maps, p->d_whi, p->d_bias,
                                   tgt_rope && tgt_rope->style == CB_ROPE_HALF_SPLIT ? 1 : 0, st) != hipSuccess)
        return fail(CB_ERR_DEVICE, "map split launch failed");
    if (N == 0) return ok();
    cb::ApplyMultiArgs a = {};
    if (src_rope) {
        if (cb_status s = ensure_rws(p, 2 * (int64_t)p->L_s * N * p->H_s * p->d_s)) return s;
        if (cb_status s = derotate_rows(src, src_rope, 1, p->d_rws, &a.ssk, st)) return s;
        a.srck = p->d_rws;
    }
    a.src = (const uint16_t *)src->data;
    a.out = (uint16_t *)tgt_out->data;
    a.ss = strides_of(src);
    a.os = strides_of(tgt_out);
    a.T = cb::make_fastdiv((uint32_t)src->seq_len);
    a.N = N;
    a.k = p->k;
    a.n_maps = p->n_maps;
    a.n_tiles = (int32_t)((N + 255) / 256);
    if ((int64_t)p->n_maps * a.n_tiles > (int64_t)INT32_MAX - 8)
        return fail(CB_ERR_UNSUPPORTED, "too many application tasks");
    a.maps = p->d_amaps;
    a.src_layers = p->d_alayers;
    a.wfrag = p->d_whi;
    a.bias = p->d_bias;
    a.rope_table = tgt_rope ? tgt_rope->table : nullptr;
    a.rope_style = tgt_rope ? tgt_rope->style : 0;
    a.rope_pos_offset = tgt_rope ? tgt_rope->pos_offset : 0;
    // pairs of maps that share their source blocks, then the maps left alone
    if (p->n_apairs > 0) {
        cb::ApplyMultiArgs ap = a;
        ap.pairs = p->d_apairs;
        ap.n_pairs = p->n_apairs;
        ap.pair_stride = p->apair_stride;
        ap.n_tasks = p->n_apairs * a.n_tiles;
        ap.per_xcd = (ap.n_tasks + 7) / 8;
        if (cb::launch_apply_multi(ap, p->n_cu, st) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer application kernel launch failed");
    }
    if (p->n_asingles > 0) {
        cb::ApplyMultiArgs as = a;
        as.pairs = nullptr;
        as.order = p->d_asingles;
        as.n_maps = p->n_asingles;
        as.n_tasks = p->n_asingles * a.n_tiles;
        as.per_xcd = (as.n_tasks + 7) / 8;
        if (cb::launch_apply_multi(as, p->n_cu, st) != hipSuccess)
            return fail(CB_ERR_DEVICE, "multi-layer application kernel launch failed");
    }
    return ok();
}

cb_status cb_apply(cb_plan *p, const float *maps, const cb_cache *src, const cb_cache *tgt_out, void *stream) {
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (p->multi) return apply_multi(p, maps, src, tgt_out, nullptr, nullptr, stream);
    return apply_single(p, maps, src, tgt_out, nullptr, nullptr, stream);
}

cb_status cb_apply_rope(cb_plan *p, const float *maps, const cb_cache *src, const cb_cache *tgt_out,
                        const cb_rope_spec *src_rope, const cb_rope_spec *tgt_rope, void *stream) {
    if (!src_rope && !tgt_rope) return cb_apply(p, maps, src, tgt_out, stream);
    if (!p) return fail(CB_ERR_INVALID_ARGUMENT, "plan is NULL");
    if (!src || !tgt_out) return fail(CB_ERR_INVALID_ARGUMENT, "src and tgt_out must be non-NULL");
    if (src_rope)
        if (cb_status s = check_rope("src_rope", src_rope, p->d_s, src->seq_len)) return s;
    if (tgt_rope)
        if (cb_status s = check_rope("tgt_rope", tgt_rope, p->d_t, src->seq_len)) return s;
    if (p->multi) return apply_multi(p, maps, src, tgt_out, src_rope, tgt_rope, stream);
    return apply_single(p, maps, src, tgt_out, src_rope, tgt_rope, stream);
}

}  // extern "C"
