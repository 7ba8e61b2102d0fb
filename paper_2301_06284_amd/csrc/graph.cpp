// graph.cpp -- host-side graph preprocessing (the COO -> CSR conversion and the
// index construction the paper emits as preprocessing code, Section "Code
// Generation"), device upload, info and export.
//
// Every order is fully specified so the arrays are reproducible bit for bit:
//   in-edges      sorted by (dst, rel, src, original edge id)
//   segments      maximal runs of equal (dst, rel) in that order
//   compact map   unique (rel, src) pairs in ascending (rel, src) order
//                 (Section "Compact Tensor Materialization": one row per pair)
//   node types    node ids stable-sorted by type (segment MM over node types)
//   out-edges     sorted in-edge positions ordered by (src, rel, position)
// All sorts are stable LSD counting sorts, O(E + N + R) each.
#include <algorithm>
#include <cstring>
#include <new>

#include "rgnn_internal.h"

namespace rgnn {

namespace {

// Stable counting sort of `perm` by key[perm[i]] in [0, K).
void counting_sort(std::vector<int32_t> &perm, const int32_t *key, int64_t K,
                   std::vector<int32_t> &tmp, std::vector<int64_t> &cnt)
{
    cnt.assign((size_t)K + 1, 0);
    for (int32_t e : perm) cnt[(size_t)key[e] + 1]++;
    for (int64_t k = 0; k < K; ++k) cnt[k + 1] += cnt[k];
    tmp.resize(perm.size());
    for (int32_t e : perm) tmp[(size_t)cnt[key[e]]++] = e;
    perm.swap(tmp);
}

}  // namespace

void build_tiles(const std::vector<int32_t> &type_ptr, int tile_rows, std::vector<Tile> &out)
{
    out.clear();
    const int ntypes = (int)type_ptr.size() - 1;
    for (int t = 0; t < ntypes; ++t)
        for (int32_t r0 = type_ptr[t]; r0 < type_ptr[t + 1]; r0 += tile_rows)
            out.push_back(Tile{t, r0, std::min<int32_t>(tile_rows, type_ptr[t + 1] - r0), 0});
}

// The rows of each relation (sorted by destination) cut where the destination
// crosses a multiple of `span` node ids, at most tile_rows rows per tile; the
// tiles of eight consecutive destination ranges are interleaved (range i of a
// group at tile positions i, i + 8, ...; empty tiles fill the gaps), so that
// the tiles of one range -- one per relation that enters it -- land on the same
// XCD (workgroups are dealt to the eight XCDs in turn) at about the same time:
// a destination row gathered by several relations' tiles is read from HBM once
// and from that XCD's L2 after that.
void build_tiles_dst_ranges(const std::vector<int32_t> &rel_ptr, const std::vector<int32_t> &row_dst, int32_t span,
                            int tile_rows, std::vector<Tile> &out)
{
    out.clear();
    const int R = (int)rel_ptr.size() - 1;
    if (R <= 0 || rel_ptr[R] == 0) return;
    struct Chunk { int32_t range, rel, row0, rows; };
    std::vector<Chunk> ch;
    for (int r = 0; r < R; ++r)
        for (int32_t i = rel_ptr[r]; i < rel_ptr[r + 1];) {
            const int32_t rg = row_dst[i] / span;
            int32_t j = i;
            while (j < rel_ptr[r + 1] && row_dst[j] / span == rg && j - i < tile_rows) ++j;
            ch.push_back(Chunk{rg, r, i, j - i});
            i = j;
        }
    // (range, relation, first row): a total order, so an in-place sort suffices
    std::sort(ch.begin(), ch.end(), [](const Chunk &a, const Chunk &b) {
        return a.range != b.range ? a.range < b.range : (a.rel != b.rel ? a.rel < b.rel : a.row0 < b.row0);
    });
    for (size_t a = 0; a < ch.size();) {
        size_t beg[8], end[8], m = 0;
        int ng = 0;
        size_t b = a;
        while (b < ch.size() && ng < 8) {
            size_t e = b;
            while (e < ch.size() && ch[e].range == ch[b].range) ++e;
            beg[ng] = b; end[ng] = e; ++ng;
            m = std::max(m, e - b);
            b = e;
        }
        for (size_t j = 0; j < m; ++j)
            for (int i = 0; i < 8; ++i) {
                if (i < ng && beg[i] + j < end[i]) {
                    const Chunk &c = ch[beg[i] + j];
                    out.push_back(Tile{c.rel, c.row0, c.rows, 0});
                } else {
                    out.push_back(Tile{0, 0, 0, 0});
                }
            }
        a = b;
    }
}

rgnn_status build_host_index(int64_t N, int32_t T, int32_t R, int64_t E, const int32_t *src,
                             const int32_t *dst, const int32_t *rel, const int32_t *ntype,
                             int32_t flags, rgnn_graph *g)
{
    const bool compact = !(flags & RGNN_GRAPH_NO_COMPACT);
    HostIndex &x = g->host;
    g->N = N; g->E = E; g->R = R; g->T = T;
    const int C = g->chunk;
    try {
        // ---- in-edges by (dst, rel, src, eid): LSD passes src, rel, dst ----
        std::vector<int32_t> perm((size_t)E), tmp;
        std::vector<int64_t> cnt;
        for (int64_t e = 0; e < E; ++e) perm[e] = (int32_t)e;
        counting_sort(perm, src, N, tmp, cnt);
        counting_sort(perm, rel, R, tmp, cnt);
        counting_sort(perm, dst, N, tmp, cnt);
        x.in_eid = perm;
        x.in_src.resize(E); x.in_rel.resize(E);
        for (int64_t i = 0; i < E; ++i) {
            x.in_src[i] = src[perm[i]];
            x.in_rel[i] = rel[perm[i]];
        }
        x.rowptr.assign((size_t)N + 1, 0);
        for (int64_t e = 0; e < E; ++e) x.rowptr[(size_t)dst[e] + 1]++;
        g->max_in_deg = 0; g->n_empty = 0;
        for (int64_t v = 0; v < N; ++v) {
            const int32_t deg = x.rowptr[v + 1];
            g->max_in_deg = std::max<int64_t>(g->max_in_deg, deg);
            g->n_empty += deg == 0;
            x.rowptr[v + 1] += x.rowptr[v];
        }
        // ---- (dst, rel) segments ----
        x.seg_ptr.clear(); x.seg_rel.clear();
        x.dst_segptr.assign((size_t)N + 1, 0);
        for (int64_t v = 0; v < N; ++v) {
            for (int32_t i = x.rowptr[v]; i < x.rowptr[v + 1]; ++i) {
                if (i == x.rowptr[v] || x.in_rel[i] != x.in_rel[i - 1]) {
                    x.seg_ptr.push_back(i);
                    x.seg_rel.push_back(x.in_rel[i]);
                }
            }
            x.dst_segptr[v + 1] = (int32_t)x.seg_ptr.size();
        }
        g->U_dst = (int64_t)x.seg_ptr.size();
        x.seg_ptr.push_back((int32_t)E);
        // ---- compact (rel, src) map: LSD passes src, rel over edge ids; without
        //      compaction every edge keeps its own row (vanilla materialization) ----
        for (int64_t e = 0; e < E; ++e) perm[e] = (int32_t)e;
        counting_sort(perm, src, N, tmp, cnt);
        counting_sort(perm, rel, R, tmp, cnt);
        std::vector<int32_t> pair_of((size_t)E);
        x.uniq_src.clear();
        x.uniq_rel_ptr.assign((size_t)R + 1, 0);
        for (int64_t i = 0; i < E; ++i) {
            const int32_t e = perm[i];
            if (!compact || i == 0 || rel[e] != rel[perm[i - 1]] || src[e] != src[perm[i - 1]]) {
                x.uniq_src.push_back(src[e]);
                x.uniq_rel_ptr[(size_t)rel[e] + 1]++;
            }
            pair_of[e] = (int32_t)x.uniq_src.size() - 1;
        }
        for (int32_t r = 0; r < R; ++r) x.uniq_rel_ptr[r + 1] += x.uniq_rel_ptr[r];
        g->U_src = (int64_t)x.uniq_src.size();
        x.e2u.resize(E);
        for (int64_t i = 0; i < E; ++i) x.e2u[i] = pair_of[x.in_eid[i]];
        // ---- node-type segments ----
        std::vector<int32_t> zeros;
        if (!ntype) { zeros.assign((size_t)N, 0); ntype = zeros.data(); }
        std::vector<int32_t> nperm((size_t)N);
        for (int64_t n = 0; n < N; ++n) nperm[n] = (int32_t)n;
        counting_sort(nperm, ntype, T, tmp, cnt);
        x.ntype_perm = nperm;
        x.ntype_ptr.assign((size_t)T + 1, 0);
        for (int64_t n = 0; n < N; ++n) x.ntype_ptr[(size_t)ntype[n] + 1]++;
        for (int32_t t = 0; t < T; ++t) x.ntype_ptr[t + 1] += x.ntype_ptr[t];
        // the destination node type of every relation (-1 when it has several;
        // a relation without edges takes type 0)
        x.rel_dsttype.assign((size_t)R, -2);
        for (int64_t e = 0; e < E; ++e) {
            int32_t &t = x.rel_dsttype[rel[e]];
            const int32_t te = ntype[dst[e]];
            t = t == -2 ? te : (t == te ? t : -1);
        }
        g->rel_dst_typed = true;
        for (int32_t r = 0; r < R; ++r) {
            if (x.rel_dsttype[r] == -2) x.rel_dsttype[r] = 0;
            if (x.rel_dsttype[r] < 0) g->rel_dst_typed = false;
        }

        // ---- virtual segments: segments cut into pieces of at most C edges ----
        x.vseg_ptr.clear(); x.vseg_rel.clear(); x.vseg_dst.clear(); x.vseg_cnt.clear(); x.vseg_seg.clear();
        x.dst_vsegptr.assign((size_t)N + 1, 0);
        x.seg_vsegptr.assign((size_t)g->U_dst + 1, 0);
        for (int64_t v = 0; v < N; ++v) {
            for (int32_t s = x.dst_segptr[v]; s < x.dst_segptr[v + 1]; ++s) {
                const int32_t b = x.seg_ptr[s], e = x.seg_ptr[s + 1];
                x.seg_vsegptr[s] = (int32_t)x.vseg_ptr.size();
                for (int32_t p = b; p < e; p += C) {
                    x.vseg_ptr.push_back(p);
                    x.vseg_rel.push_back(x.seg_rel[s]);
                    x.vseg_dst.push_back((int32_t)v);
                    x.vseg_cnt.push_back(e - b);
                    x.vseg_seg.push_back(s);
                }
            }
            x.dst_vsegptr[v + 1] = (int32_t)x.vseg_ptr.size();
        }
        g->V = (int64_t)x.vseg_ptr.size();
        x.vseg_ptr.push_back((int32_t)E);
        x.seg_vsegptr[(size_t)g->U_dst] = (int32_t)g->V;
        x.big_seg.clear();
        for (int64_t sg = 0; sg < g->U_dst; ++sg)
            if (x.seg_vsegptr[sg + 1] - x.seg_vsegptr[sg] > kBigRange) x.big_seg.push_back((int32_t)sg);
        g->n_big_seg = (int64_t)x.big_seg.size();
        // vsegs grouped by relation (stable: (rel, dst) order) for the typed GEMMs
        std::vector<int32_t> vperm((size_t)g->V);
        for (int64_t i = 0; i < g->V; ++i) vperm[i] = (int32_t)i;
        counting_sort(vperm, x.vseg_rel.data(), R, tmp, cnt);
        x.vseg_byrel = vperm;
        x.rel_vsegptr.assign((size_t)R + 1, 0);
        for (int64_t i = 0; i < g->V; ++i) x.rel_vsegptr[(size_t)x.vseg_rel[i] + 1]++;
        for (int32_t r = 0; r < R; ++r) x.rel_vsegptr[r + 1] += x.rel_vsegptr[r];
        x.vsegdst_byrel.resize((size_t)g->V);
        for (int64_t i = 0; i < g->V; ++i) x.vsegdst_byrel[i] = x.vseg_dst[x.vseg_byrel[i]];
        x.invcnt_byrel.resize((size_t)g->V);
        for (int64_t i = 0; i < g->V; ++i) x.invcnt_byrel[i] = 1.f / (float)x.vseg_cnt[x.vseg_byrel[i]];
        // fused aggregate-first order: by relation, then edge count (largest
        // first), then id; tiles of consecutive rows of one relation, cut at
        // kFusedTileRows rows or (after the first 16-row block) kFusedTileEdges
        // edges
        {
            std::vector<int32_t> fperm((size_t)g->V), fkey((size_t)g->V);
            for (int64_t i = 0; i < g->V; ++i) {
                fperm[i] = (int32_t)i;
                fkey[i] = C - (x.vseg_ptr[i + 1] - x.vseg_ptr[i]);
            }
            counting_sort(fperm, fkey.data(), C, tmp, cnt);
            counting_sort(fperm, x.vseg_rel.data(), R, tmp, cnt);
            x.fused_rows.resize((size_t)g->V);
            x.fused_src.resize((size_t)E);
            x.vseg_fpos.resize((size_t)g->V);
            int32_t fpos = 0;
            for (int64_t i = 0; i < g->V; ++i) {
                const int32_t vs = fperm[i];
                const int32_t b = x.vseg_ptr[vs], n = x.vseg_ptr[vs + 1] - b;
                const int32_t v = x.vseg_dst[vs];
                const bool only = x.dst_vsegptr[(size_t)v + 1] - x.dst_vsegptr[v] == 1;
                x.fused_rows[i] = FusedRow{vs, fpos, n, only ? ~v : x.vseg_cnt[vs]};
                x.vseg_fpos[vs] = (int32_t)i;
                for (int32_t j = 0; j < n; ++j) x.fused_src[(size_t)fpos + j] = x.in_src[(size_t)b + j];
                fpos += n;
            }
            x.tiles_fused.clear();
            for (int32_t r = 0; r < R; ++r) {
                const int32_t end = x.rel_vsegptr[r + 1];
                int32_t r0 = x.rel_vsegptr[r];
                while (r0 < end) {
                    int32_t rows = 0, edges = 0;
                    while (rows < kFusedTileRows && r0 + rows < end) {
                        const int32_t nb = std::min<int32_t>(16, end - (r0 + rows));
                        int32_t be = 0;
                        for (int32_t j = 0; j < nb; ++j) be += x.fused_rows[r0 + rows + j].ne;
                        if (rows > 0 && edges + be > kFusedTileEdges) break;
                        rows += nb;
                        edges += be;
                    }
                    x.tiles_fused.push_back(Tile{r, r0, rows, x.fused_rows[r0].e0});
                    r0 += rows;
                }
            }
            g->n_tiles_fused = (int64_t)x.tiles_fused.size();
        }

        // ---- traversal work items ----
        x.items.clear(); x.item_slot.clear(); x.split_dst.clear();
        x.split_slotptr.assign(1, 0);
        int32_t slots = 0;
        int64_t v = 0;
        auto deg = [&](int64_t u) { return x.rowptr[u + 1] - x.rowptr[u]; };
        while (v < N) {
            if (deg(v) > C) {
                int32_t s = x.dst_vsegptr[v];
                const int32_t se = x.dst_vsegptr[v + 1];
                while (s < se) {
                    const int32_t s0 = s;
                    int32_t tot = 0;
                    while (s < se && (s == s0 || tot + (x.vseg_ptr[s + 1] - x.vseg_ptr[s]) <= C)) {
                        tot += x.vseg_ptr[s + 1] - x.vseg_ptr[s];
                        ++s;
                    }
                    x.items.push_back(Item{(int32_t)v, (int32_t)v + 1, s0, s});
                    x.item_slot.push_back(slots++);
                }
                x.split_dst.push_back((int32_t)v);
                x.split_slotptr.push_back(slots);
                ++v;
            } else {
                const int64_t v0 = v;
                int64_t tot = 0;
                while (v < N && deg(v) <= C && tot + deg(v) <= C && v - v0 < kMaxDstPerItem) {
                    tot += deg(v);
                    ++v;
                }
                x.items.push_back(Item{(int32_t)v0, (int32_t)v, x.dst_vsegptr[v0], x.dst_vsegptr[v]});
                x.item_slot.push_back(-1);
            }
        }
        g->n_items = (int64_t)x.items.size();
        x.split_items.clear();
        for (int64_t i = 0; i < g->n_items; ++i)
            if (x.item_slot[i] >= 0) x.split_items.push_back((int32_t)i);
        g->n_split_items = (int64_t)x.split_items.size();
        g->n_split = (int64_t)x.split_dst.size();
        g->n_slots = slots;
        x.big_split.clear();
        for (int64_t i = 0; i < g->n_split; ++i)
            if (x.split_slotptr[i + 1] - x.split_slotptr[i] > kBigRange) x.big_split.push_back((int32_t)i);
        x.big_chunkptr.assign(1, 0);
        x.chunk_lo.clear(); x.chunk_hi.clear();
        for (int32_t i : x.big_split) {
            for (int32_t sl = x.split_slotptr[i]; sl < x.split_slotptr[i + 1]; sl += kMergeChunk) {
                x.chunk_lo.push_back(sl);
                x.chunk_hi.push_back(std::min<int32_t>(sl + kMergeChunk, x.split_slotptr[i + 1]));
            }
            x.big_chunkptr.push_back((int32_t)x.chunk_lo.size());
        }
        g->n_big_chunks = (int64_t)x.chunk_lo.size();
        auto order_by_slots = [](const std::vector<int32_t> &ptr, std::vector<int32_t> &order, int64_t &nwide) {
            const int64_t n = (int64_t)ptr.size() - 1;
            order.resize((size_t)n);
            for (int64_t i = 0; i < n; ++i) order[i] = (int32_t)i;
            std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {   // ties in index order
                const int32_t na = ptr[a + 1] - ptr[a], nb = ptr[b + 1] - ptr[b];
                return na != nb ? na > nb : a < b;
            });
            nwide = 0;
            while (nwide < n && ptr[order[nwide] + 1] - ptr[order[nwide]] > kWaveSlots) ++nwide;
        };
        order_by_slots(x.split_slotptr, x.split_order, g->n_split_wide);
        // destinations with many segments, largest first (ties in id order):
        // their reductions take whole workgroups at the front of the grid
        x.big_vdst.clear();
        for (int64_t u = 0; u < N; ++u)
            if (x.dst_vsegptr[u + 1] - x.dst_vsegptr[u] > kBigRange) x.big_vdst.push_back((int32_t)u);
        std::stable_sort(x.big_vdst.begin(), x.big_vdst.end(), [&](int32_t a, int32_t b) {
            return x.dst_vsegptr[a + 1] - x.dst_vsegptr[a] > x.dst_vsegptr[b + 1] - x.dst_vsegptr[b];
        });
        g->n_big_split = (int64_t)x.big_split.size();
        g->n_big_vdst = (int64_t)x.big_vdst.size();
        // destinations a segment reduction still visits when the fused kernel
        // finishes those with a single virtual segment (the rest up to
        // kBigRange segments, empty ones included), in id order
        x.reduce_dst.clear();
        for (int64_t u = 0; u < N; ++u) {
            const int32_t n = x.dst_vsegptr[u + 1] - x.dst_vsegptr[u];
            if (n != 1 && n <= kBigRange) x.reduce_dst.push_back((int32_t)u);
        }
        g->n_reduce_dst = (int64_t)x.reduce_dst.size();

        // ---- out-edges: in-edge positions by (src, rel, position) ----
        {
            std::vector<int32_t> pos((size_t)E);
            for (int64_t i = 0; i < E; ++i) pos[i] = (int32_t)i;
            counting_sort(pos, x.in_rel.data(), R, tmp, cnt);
            counting_sort(pos, x.in_src.data(), N, tmp, cnt);
            x.out_pos = pos;
            x.out_ptr.assign((size_t)N + 1, 0);
            for (int64_t i = 0; i < E; ++i) x.out_ptr[(size_t)x.in_src[i] + 1]++;
            for (int64_t u = 0; u < N; ++u) x.out_ptr[u + 1] += x.out_ptr[u];
            std::vector<int32_t> pos_vseg((size_t)E);
            for (int64_t vs = 0; vs < g->V; ++vs)
                for (int32_t i = x.vseg_ptr[vs]; i < x.vseg_ptr[vs + 1]; ++i) pos_vseg[i] = (int32_t)vs;
            // out_vseg holds the by-relation position of the in-edge's vseg
            x.vseg_pos.resize((size_t)g->V);
            for (int64_t i = 0; i < g->V; ++i) x.vseg_pos[x.vseg_byrel[i]] = (int32_t)i;
            x.out_vseg.resize((size_t)E);
            x.out_rel.resize((size_t)E);
            x.out_pair.resize((size_t)E);
            x.out_vs.resize((size_t)E);
            x.out_dst.resize((size_t)E);
            for (int64_t q = 0; q < E; ++q) {
                x.out_vseg[q] = x.vseg_pos[pos_vseg[x.out_pos[q]]];
                x.out_rel[q] = x.in_rel[x.out_pos[q]];
                x.out_pair[q] = x.e2u[x.out_pos[q]];
                x.out_vs[q] = pos_vseg[x.out_pos[q]];
                x.out_dst[q] = x.vseg_dst[x.out_vs[q]];
            }
            // work items over out-edges: bundles of small sources, pieces of large ones
            x.oitems.clear();
            x.osplit.clear();
            x.oitem_slot.clear();
            x.osplit_slotptr.assign(1, 0);
            auto odeg = [&](int64_t u) { return x.out_ptr[u + 1] - x.out_ptr[u]; };
            int64_t u = 0;
            while (u < N) {
                if (odeg(u) > C) {
                    x.osplit.push_back((int32_t)u);
                    for (int32_t q = x.out_ptr[u]; q < x.out_ptr[u + 1]; q += C) {
                        x.oitems.push_back(Item{(int32_t)u, (int32_t)u + 1, q,
                                                std::min<int32_t>(q + C, x.out_ptr[u + 1])});
                        x.oitem_slot.push_back(x.osplit_slotptr.back() + (q - x.out_ptr[u]) / C);
                    }
                    x.osplit_slotptr.push_back(x.osplit_slotptr.back() + (odeg(u) + C - 1) / C);
                    ++u;
                } else {
                    const int64_t u0 = u;
                    int64_t tot = 0;
                    while (u < N && odeg(u) <= C && tot + odeg(u) <= C && u - u0 < kMaxDstPerItem) {
                        tot += odeg(u);
                        ++u;
                    }
                    x.oitems.push_back(Item{(int32_t)u0, (int32_t)u, x.out_ptr[u0], x.out_ptr[u]});
                    x.oitem_slot.push_back(-1);
                }
            }
            g->n_oitems = (int64_t)x.oitems.size();
            g->n_osplit = (int64_t)x.osplit.size();
            g->n_oslots = x.osplit_slotptr.back();
            order_by_slots(x.osplit_slotptr, x.osplit_order, g->n_osplit_wide);
        }

        // ---- GEMM tile tables ----
        build_tiles(x.uniq_rel_ptr, kGemmTileRows, x.tiles_pairs);
        build_tiles(x.rel_vsegptr, kGemmTileRows, x.tiles_vsegs);
        build_tiles_dst_ranges(x.rel_vsegptr, x.vsegdst_byrel, kGemmTileRows, kGemmTileRows, x.tiles_vsegs_dst);
        g->n_tiles_vsegs_dst = (int64_t)x.tiles_vsegs_dst.size();
        build_tiles(x.ntype_ptr, kGemmTileRows, x.tiles_nodes);
        std::vector<int32_t> all{0, (int32_t)N};
        build_tiles(all, kGemmTileRows, x.tiles_all);
        g->n_tiles_pairs = (int64_t)x.tiles_pairs.size();
        g->n_tiles_vsegs = (int64_t)x.tiles_vsegs.size();
        g->n_tiles_nodes = (int64_t)x.tiles_nodes.size();
        g->n_tiles_all = (int64_t)x.tiles_all.size();
        build_tiles(x.rel_vsegptr, kOuterRows, x.tiles_outer);
        g->n_tiles_outer = (int64_t)x.tiles_outer.size();
        build_tiles(all, kOuterRows, x.tiles_nodes_outer);   // node chunks (self-loop dW0)
        g->n_tiles_nodes_outer = (int64_t)x.tiles_nodes_outer.size();
        x.nodes_chunkptr = {0, (int32_t)g->n_tiles_nodes_outer};
        // chunks over the nodes grouped by type (per-type weight gradients)
        build_tiles(x.ntype_ptr, kOuterRows, x.tiles_types_outer);
        g->n_tiles_types_outer = (int64_t)x.tiles_types_outer.size();
        x.types_chunkptr.assign((size_t)T + 1, 0);
        for (const Tile &t : x.tiles_types_outer) x.types_chunkptr[(size_t)t.type + 1]++;
        for (int32_t t = 0; t < T; ++t) x.types_chunkptr[t + 1] += x.types_chunkptr[t];
        x.rel_chunkptr.assign((size_t)R + 1, 0);
        for (const Tile &t : x.tiles_outer) x.rel_chunkptr[(size_t)t.type + 1]++;
        for (int32_t r = 0; r < R; ++r) x.rel_chunkptr[r + 1] += x.rel_chunkptr[r];
        x.rel_pairtileptr.assign((size_t)R + 1, 0);
        for (const Tile &t : x.tiles_pairs) x.rel_pairtileptr[(size_t)t.type + 1]++;
        for (int32_t r = 0; r < R; ++r) x.rel_pairtileptr[r + 1] += x.rel_pairtileptr[r];
        // outer-product chunks over the pairs of each relation
        build_tiles(x.uniq_rel_ptr, kOuterRows, x.tiles_outer_pairs);
        g->n_tiles_outer_pairs = (int64_t)x.tiles_outer_pairs.size();
        x.rel_pairchunkptr.assign((size_t)R + 1, 0);
        for (const Tile &t : x.tiles_outer_pairs) x.rel_pairchunkptr[(size_t)t.type + 1]++;
        for (int32_t r = 0; r < R; ++r) x.rel_pairchunkptr[r + 1] += x.rel_pairchunkptr[r];
        // compact pairs in source-major order: a stable pass by source over the
        // (rel, src) order gives (src, rel)
        {
            std::vector<int32_t> pp((size_t)g->U_src);
            for (int64_t i = 0; i < g->U_src; ++i) pp[i] = (int32_t)i;
            counting_sort(pp, x.uniq_src.data(), N, tmp, cnt);
            x.pair_smpos.resize((size_t)g->U_src);
            for (int64_t i = 0; i < g->U_src; ++i) x.pair_smpos[pp[i]] = (int32_t)i;
            x.src_pairptr.assign((size_t)N + 1, 0);
            for (int64_t i = 0; i < g->U_src; ++i) x.src_pairptr[(size_t)x.uniq_src[i] + 1]++;
            for (int64_t u = 0; u < N; ++u) x.src_pairptr[u + 1] += x.src_pairptr[u];
        }
        // virtual pairs: a pair's out-edges are consecutive in the out-edge
        // order (src, rel, position); pieces of at most kPairPiece of them, per
        // relation ordered by out-edge count (most first, then by source), so
        // that the pairs a workgroup gathers together have similar counts;
        // then their rows in source-major order and chunks per relation
        {
            std::vector<int32_t> oe0((size_t)g->U_src, -1), oen((size_t)g->U_src, 0);
            for (int64_t q = 0; q < E; ++q) {
                const int32_t p = x.out_pair[q];
                if (oe0[p] < 0) oe0[p] = (int32_t)q;
                oen[p]++;
            }
            x.vpair_oe0.clear(); x.vpair_ne.clear(); x.vpair_src.clear();
            std::vector<int32_t> rel_vpairptr((size_t)R + 1, 0);
            std::vector<int32_t> bucket_cnt((size_t)kPairPiece + 2, 0);
            for (int32_t r = 0; r < R; ++r) {
                // counting sort of the relation's pieces by descending count
                std::fill(bucket_cnt.begin(), bucket_cnt.end(), 0);
                for (int32_t p = x.uniq_rel_ptr[r]; p < x.uniq_rel_ptr[r + 1]; ++p)
                    for (int32_t o = 0; o < oen[p]; o += kPairPiece)
                        bucket_cnt[(size_t)(kPairPiece - std::min<int32_t>(kPairPiece, oen[p] - o)) + 1]++;
                for (int32_t b = 0; b <= kPairPiece; ++b) bucket_cnt[(size_t)b + 1] += bucket_cnt[b];
                const size_t base = x.vpair_src.size();
                const size_t n = base + (size_t)bucket_cnt[(size_t)kPairPiece + 1];
                x.vpair_oe0.resize(n); x.vpair_ne.resize(n); x.vpair_src.resize(n);
                for (int32_t p = x.uniq_rel_ptr[r]; p < x.uniq_rel_ptr[r + 1]; ++p)
                    for (int32_t o = 0; o < oen[p]; o += kPairPiece) {
                        const int32_t ne = std::min<int32_t>(kPairPiece, oen[p] - o);
                        const size_t at = base + (size_t)bucket_cnt[(size_t)(kPairPiece - ne)]++;
                        x.vpair_oe0[at] = oe0[p] + o;
                        x.vpair_ne[at] = ne;
                        x.vpair_src[at] = x.uniq_src[p];
                    }
                rel_vpairptr[(size_t)r + 1] = (int32_t)x.vpair_src.size();
            }
            g->n_vpairs = (int64_t)x.vpair_src.size();
            std::vector<int32_t> vp((size_t)g->n_vpairs);
            for (int64_t i = 0; i < g->n_vpairs; ++i) vp[i] = (int32_t)i;
            counting_sort(vp, x.vpair_src.data(), N, tmp, cnt);
            x.vpair_smpos.resize((size_t)g->n_vpairs);
            for (int64_t i = 0; i < g->n_vpairs; ++i) x.vpair_smpos[vp[i]] = (int32_t)i;
            x.src_vpairptr.assign((size_t)N + 1, 0);
            for (int64_t i = 0; i < g->n_vpairs; ++i) x.src_vpairptr[(size_t)x.vpair_src[i] + 1]++;
            for (int64_t u = 0; u < N; ++u) x.src_vpairptr[u + 1] += x.src_vpairptr[u];
            build_tiles(rel_vpairptr, kPairChunkRows, x.tiles_vpairs);
            g->n_tiles_vpairs = (int64_t)x.tiles_vpairs.size();
            x.rel_vpairchunkptr.assign((size_t)R + 1, 0);
            for (const Tile &t : x.tiles_vpairs) x.rel_vpairchunkptr[(size_t)t.type + 1]++;
            for (int32_t r = 0; r < R; ++r) x.rel_vpairchunkptr[r + 1] += x.rel_vpairchunkptr[r];
        }
    } catch (const std::bad_alloc &) {
        return fail(RGNN_ENOMEM, "host allocation failed while building the graph index");
    }
    return RGNN_OK;
}

namespace {

template <class T>
size_t padded(size_t n) { return (n * sizeof(T) + 255) & ~size_t(255); }

rgnn_status upload(rgnn_graph *g, hipStream_t s)
{
    HostIndex &x = g->host;
    DeviceIndex &d = g->dev;
    struct Part { void **dst; const void *src; size_t bytes; };
    std::vector<Part> parts;
    auto add32 = [&](int32_t **p, const std::vector<int32_t> &v) {
        parts.push_back(Part{(void **)p, v.data(), v.size() * sizeof(int32_t)});
    };
    add32(&d.rowptr, x.rowptr); add32(&d.in_src, x.in_src); add32(&d.in_rel, x.in_rel);
    add32(&d.in_eid, x.in_eid); add32(&d.seg_ptr, x.seg_ptr); add32(&d.seg_rel, x.seg_rel);
    add32(&d.dst_segptr, x.dst_segptr); add32(&d.uniq_src, x.uniq_src);
    add32(&d.uniq_rel_ptr, x.uniq_rel_ptr); add32(&d.e2u, x.e2u);
    add32(&d.ntype_perm, x.ntype_perm); add32(&d.ntype_ptr, x.ntype_ptr); add32(&d.rel_dsttype, x.rel_dsttype);
    add32(&d.vseg_ptr, x.vseg_ptr); add32(&d.vseg_rel, x.vseg_rel); add32(&d.vseg_dst, x.vseg_dst);
    add32(&d.vseg_cnt, x.vseg_cnt); add32(&d.dst_vsegptr, x.dst_vsegptr);
    add32(&d.vseg_byrel, x.vseg_byrel); add32(&d.rel_vsegptr, x.rel_vsegptr);
    add32(&d.vsegdst_byrel, x.vsegdst_byrel); add32(&d.rel_chunkptr, x.rel_chunkptr);
    add32(&d.rel_pairtileptr, x.rel_pairtileptr);
    add32(&d.item_slot, x.item_slot); add32(&d.split_dst, x.split_dst); add32(&d.split_items, x.split_items);
    add32(&d.split_slotptr, x.split_slotptr);
    add32(&d.big_split, x.big_split); add32(&d.big_vdst, x.big_vdst); add32(&d.reduce_dst, x.reduce_dst);
    add32(&d.big_chunkptr, x.big_chunkptr); add32(&d.chunk_lo, x.chunk_lo); add32(&d.chunk_hi, x.chunk_hi);
    add32(&d.seg_vsegptr, x.seg_vsegptr); add32(&d.big_seg, x.big_seg); add32(&d.osplit, x.osplit);
    add32(&d.oitem_slot, x.oitem_slot); add32(&d.osplit_slotptr, x.osplit_slotptr);
    add32(&d.split_order, x.split_order); add32(&d.osplit_order, x.osplit_order);
    parts.push_back(Part{(void **)&d.items, x.items.data(), x.items.size() * sizeof(Item)});
    parts.push_back(Part{(void **)&d.tiles_pairs, x.tiles_pairs.data(), x.tiles_pairs.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_vsegs, x.tiles_vsegs.data(), x.tiles_vsegs.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_vsegs_dst, x.tiles_vsegs_dst.data(),
                         x.tiles_vsegs_dst.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_nodes, x.tiles_nodes.data(), x.tiles_nodes.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_all, x.tiles_all.data(), x.tiles_all.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_outer, x.tiles_outer.data(), x.tiles_outer.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.tiles_nodes_outer, x.tiles_nodes_outer.data(),
                         x.tiles_nodes_outer.size() * sizeof(Tile)});
    add32(&d.nodes_chunkptr, x.nodes_chunkptr);
    parts.push_back(Part{(void **)&d.tiles_types_outer, x.tiles_types_outer.data(),
                         x.tiles_types_outer.size() * sizeof(Tile)});
    add32(&d.types_chunkptr, x.types_chunkptr);
    parts.push_back(Part{(void **)&d.invcnt_byrel, x.invcnt_byrel.data(), x.invcnt_byrel.size() * sizeof(float)});
    parts.push_back(Part{(void **)&d.tiles_fused, x.tiles_fused.data(), x.tiles_fused.size() * sizeof(Tile)});
    parts.push_back(Part{(void **)&d.fused_rows, x.fused_rows.data(), x.fused_rows.size() * sizeof(FusedRow)});
    add32(&d.fused_src, x.fused_src);
    add32(&d.vseg_fpos, x.vseg_fpos);
    add32(&d.vseg_seg, x.vseg_seg);
    add32(&d.out_ptr, x.out_ptr); add32(&d.out_pos, x.out_pos); add32(&d.out_vseg, x.out_vseg);
    add32(&d.out_rel, x.out_rel); add32(&d.vseg_pos, x.vseg_pos); add32(&d.out_pair, x.out_pair);
    add32(&d.out_vs, x.out_vs); add32(&d.out_dst, x.out_dst);
    parts.push_back(Part{(void **)&d.oitems, x.oitems.data(), x.oitems.size() * sizeof(Item)});
    add32(&d.src_pairptr, x.src_pairptr); add32(&d.pair_smpos, x.pair_smpos);
    add32(&d.rel_pairchunkptr, x.rel_pairchunkptr);
    parts.push_back(Part{(void **)&d.tiles_outer_pairs, x.tiles_outer_pairs.data(),
                         x.tiles_outer_pairs.size() * sizeof(Tile)});
    add32(&d.vpair_oe0, x.vpair_oe0); add32(&d.vpair_ne, x.vpair_ne); add32(&d.vpair_src, x.vpair_src);
    add32(&d.vpair_smpos, x.vpair_smpos); add32(&d.src_vpairptr, x.src_vpairptr);
    add32(&d.rel_vpairchunkptr, x.rel_vpairchunkptr);
    parts.push_back(Part{(void **)&d.tiles_vpairs, x.tiles_vpairs.data(), x.tiles_vpairs.size() * sizeof(Tile)});
    size_t total = 0;
    for (auto &p : parts) total += (p.bytes + 255) & ~size_t(255);
    total = std::max<size_t>(total, 256);
    hipError_t e = hipMalloc(&d.base, total);
    if (e != hipSuccess) {
        d.base = nullptr;
        return e == hipErrorOutOfMemory ? fail(RGNN_ENOMEM, "hipMalloc of the graph index failed")
                                        : hip_fail(e, "hipMalloc");
    }
    d.bytes = total;
    size_t off = 0;
    for (auto &p : parts) {
        *p.dst = (char *)d.base + off;
        if (p.bytes) {
            e = hipMemcpyAsync(*p.dst, p.src, p.bytes, hipMemcpyHostToDevice, s);
            if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (graph upload)");
        }
        off += (p.bytes + 255) & ~size_t(255);
    }
    e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize (graph upload)");
    return RGNN_OK;
}

rgnn_status create_common(int64_t N, int32_t T, int32_t R, int64_t E, const int32_t *src,
                          const int32_t *dst, const int32_t *rel, const int32_t *ntype,
                          int32_t flags, void *stream, rgnn_graph_t **out)
{
    if (!out) return fail(RGNN_EINVAL, "out is NULL");
    *out = nullptr;
    if (N < 0 || E < 0) return fail(RGNN_EINVAL, "negative node or edge count");
    if (N >= (int64_t(1) << 31) - 1 || E >= (int64_t(1) << 31) - 1)
        return fail(RGNN_ERANGE, "node and edge counts must be below 2^31 - 1");
    if (R <= 0 || T <= 0) return fail(RGNN_EINVAL, "num_rels and num_ntypes must be positive");
    if (E > 0 && (!src || !dst || !rel)) return fail(RGNN_EINVAL, "NULL edge array");
    if (flags & ~(RGNN_GRAPH_HOST_ONLY | RGNN_GRAPH_NO_COMPACT)) return fail(RGNN_EINVAL, "unknown graph flag");
    for (int64_t e = 0; e < E; ++e) {
        if (src[e] < 0 || src[e] >= N || dst[e] < 0 || dst[e] >= N)
            return fail(RGNN_ERANGE, "edge " + std::to_string(e) + ": node id out of range");
        if (rel[e] < 0 || rel[e] >= R)
            return fail(RGNN_ERANGE, "edge " + std::to_string(e) + ": relation out of range");
    }
    if (ntype)
        for (int64_t n = 0; n < N; ++n)
            if (ntype[n] < 0 || ntype[n] >= T)
                return fail(RGNN_ERANGE, "node " + std::to_string(n) + ": node type out of range");
    rgnn_graph *g = new (std::nothrow) rgnn_graph();
    if (!g) return fail(RGNN_ENOMEM, "host allocation failed");
    rgnn_status st = build_host_index(N, T, R, E, src, dst, rel, ntype, flags, g);
    if (st != RGNN_OK) { delete g; return st; }
    if (!(flags & RGNN_GRAPH_HOST_ONLY)) {
        int dev = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) { delete g; return hip_fail(e, "hipGetDevice"); }
        g->device = dev;
        st = upload(g, (hipStream_t)stream);
        if (st != RGNN_OK) {
            if (g->dev.base) (void)hipFree(g->dev.base);
            delete g;
            return st;
        }
        // The device copy is authoritative; drop the large host arrays.
        HostIndex empty;
        g->host.in_src.swap(empty.in_src); g->host.in_rel.swap(empty.in_rel);
        g->host.in_eid.swap(empty.in_eid); g->host.e2u.swap(empty.e2u);
        g->host.out_pos.swap(empty.out_pos); g->host.out_vseg.swap(empty.out_vseg);
        g->host.out_rel.swap(empty.out_rel); g->host.out_pair.swap(empty.out_pair);
        g->host.out_vs.swap(empty.out_vs); g->host.out_dst.swap(empty.out_dst);
        g->host.vpair_oe0.swap(empty.vpair_oe0); g->host.vpair_ne.swap(empty.vpair_ne);
        g->host.vpair_src.swap(empty.vpair_src); g->host.vpair_smpos.swap(empty.vpair_smpos);
    }
    *out = g;
    return RGNN_OK;
}

}  // namespace
}  // namespace rgnn

using namespace rgnn;

extern "C" rgnn_status rgnn_graph_create_coo(int64_t num_nodes, int32_t num_ntypes,
                                             int32_t num_rels, int64_t num_edges,
                                             const int32_t *src, const int32_t *dst,
                                             const int32_t *rel, const int32_t *ntype,
                                             int32_t flags, void *stream, rgnn_graph_t **out)
{
    return create_common(num_nodes, num_ntypes, num_rels, num_edges, src, dst, rel, ntype, flags,
                         stream, out);
}

extern "C" rgnn_status rgnn_graph_create_csr(int64_t num_nodes, int32_t num_ntypes,
                                             int32_t num_rels, const int64_t *dst_rowptr,
                                             const int32_t *col_src, const int32_t *rel,
                                             const int32_t *ntype, int32_t flags, void *stream,
                                             rgnn_graph_t **out)
{
    if (!out) return fail(RGNN_EINVAL, "out is NULL");
    *out = nullptr;
    if (num_nodes < 0) return fail(RGNN_EINVAL, "negative node count");
    if (!dst_rowptr) return fail(RGNN_EINVAL, "dst_rowptr is NULL");
    if (dst_rowptr[0] != 0) return fail(RGNN_EINVAL, "dst_rowptr[0] must be 0");
    for (int64_t v = 0; v < num_nodes; ++v)
        if (dst_rowptr[v + 1] < dst_rowptr[v])
            return fail(RGNN_EINVAL, "dst_rowptr is not monotone at " + std::to_string(v));
    const int64_t E = dst_rowptr[num_nodes];
    if (E >= (int64_t(1) << 31) - 1) return fail(RGNN_ERANGE, "edge count must be below 2^31 - 1");
    std::vector<int32_t> dst;
    try {
        dst.resize((size_t)E);
    } catch (const std::bad_alloc &) {
        return fail(RGNN_ENOMEM, "host allocation failed");
    }
    for (int64_t v = 0; v < num_nodes; ++v)
        for (int64_t i = dst_rowptr[v]; i < dst_rowptr[v + 1]; ++i) dst[i] = (int32_t)v;
    return create_common(num_nodes, num_ntypes, num_rels, E, col_src, dst.data(), rel, ntype,
                         flags, stream, out);
}

extern "C" rgnn_status rgnn_graph_destroy(rgnn_graph_t *g)
{
    if (!g) return RGNN_OK;
    if (g->dev.base) {
        int cur = 0;
        (void)hipGetDevice(&cur);
        if (cur != g->device) (void)hipSetDevice(g->device);
        hipError_t e = hipFree(g->dev.base);
        if (cur != g->device) (void)hipSetDevice(cur);
        g->dev.base = nullptr;
        if (e != hipSuccess) { delete g; return hip_fail(e, "hipFree"); }
    }
    delete g;
    return RGNN_OK;
}

extern "C" rgnn_status rgnn_graph_info(const rgnn_graph_t *g, rgnn_graph_info_t *info)
{
    if (!g || !info) return fail(RGNN_EINVAL, "NULL argument");
    info->num_nodes = g->N;
    info->num_edges = g->E;
    info->num_rels = g->R;
    info->num_ntypes = g->T;
    info->num_src_pairs = g->U_src;
    info->num_dst_segments = g->U_dst;
    info->max_in_degree = g->max_in_deg;
    info->num_empty_dst = g->n_empty;
    info->num_vsegs = g->V;
    info->num_items = g->n_items;
    info->num_split_dst = g->n_split;
    info->chunk_edges = g->chunk;
    info->device = g->device;
    return RGNN_OK;
}

extern "C" rgnn_status rgnn_graph_export(const rgnn_graph_t *g, int32_t kind, void *dst,
                                         size_t bytes)
{
    if (!g || !dst) return fail(RGNN_EINVAL, "NULL argument");
    const HostIndex &x = g->host;
    const DeviceIndex &d = g->dev;
    const std::vector<int32_t> *hv = nullptr;
    const int32_t *dp = nullptr;
    size_t n = 0;
    switch (kind) {
    case RGNN_IDX_DST_ROWPTR: hv = &x.rowptr; dp = d.rowptr; n = (size_t)g->N + 1; break;
    case RGNN_IDX_IN_SRC: hv = &x.in_src; dp = d.in_src; n = (size_t)g->E; break;
    case RGNN_IDX_IN_REL: hv = &x.in_rel; dp = d.in_rel; n = (size_t)g->E; break;
    case RGNN_IDX_IN_EID: hv = &x.in_eid; dp = d.in_eid; n = (size_t)g->E; break;
    case RGNN_IDX_SEG_PTR: hv = &x.seg_ptr; dp = d.seg_ptr; n = (size_t)g->U_dst + 1; break;
    case RGNN_IDX_SEG_REL: hv = &x.seg_rel; dp = d.seg_rel; n = (size_t)g->U_dst; break;
    case RGNN_IDX_DST_SEGPTR: hv = &x.dst_segptr; dp = d.dst_segptr; n = (size_t)g->N + 1; break;
    case RGNN_IDX_UNIQ_SRC: hv = &x.uniq_src; dp = d.uniq_src; n = (size_t)g->U_src; break;
    case RGNN_IDX_UNIQ_REL_PTR: hv = &x.uniq_rel_ptr; dp = d.uniq_rel_ptr; n = (size_t)g->R + 1; break;
    case RGNN_IDX_EDGE2UNIQ: hv = &x.e2u; dp = d.e2u; n = (size_t)g->E; break;
    case RGNN_IDX_NTYPE_PERM: hv = &x.ntype_perm; dp = d.ntype_perm; n = (size_t)g->N; break;
    case RGNN_IDX_NTYPE_PTR: hv = &x.ntype_ptr; dp = d.ntype_ptr; n = (size_t)g->T + 1; break;
    case RGNN_IDX_OUT_PTR: hv = &x.out_ptr; dp = d.out_ptr; n = (size_t)g->N + 1; break;
    case RGNN_IDX_OUT_POS: hv = &x.out_pos; dp = d.out_pos; n = (size_t)g->E; break;
    default: return fail(RGNN_EINVAL, "unknown index kind " + std::to_string(kind));
    }
    if (bytes < n * sizeof(int32_t))
        return fail(RGNN_EINVAL, "export buffer too small: need " +
                                     std::to_string(n * sizeof(int32_t)) + " bytes");
    if (n == 0) return RGNN_OK;
    if (g->device < 0) {
        std::memcpy(dst, hv->data(), n * sizeof(int32_t));
        return RGNN_OK;
    }
    hipError_t e = hipMemcpy(dst, dp, n * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy (export)");
    return RGNN_OK;
}
