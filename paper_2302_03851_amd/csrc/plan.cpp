// Batching-aware arena plan (Section 3.1 of ED-Batch: source and result
// operands of every batch should be contiguous and aligned, otherwise a
// gather or scatter runs around the batch).
//
// Runtime reading of the layout problem: a single reverse pass over the
// schedule in which consumers claim consecutive slots for their operand lists
// before the producers are placed.
//   for b = B-1 .. 0:
//     order_b = batch b stably sorted by slot (unset last); unset nodes take
//               the next slots in that order (this makes results contiguous
//               whenever a consumer claimed them as one fresh list)
//     operand lists: one per positional child p, then the ragged list
//     a list whose present entries are all unset and distinct is "fresh":
//       absent entries take a new zero pad slot, nodes the next slot, in
//       list order, so the list becomes contiguous;
//     otherwise unset entries take the next slots and absent entries read
//       the zero row (slot 0).
// Every slot a batch reads or writes is final once the batch is processed,
// so its descriptors are emitted in the same pass.  Slot 0 is the zero row.
// x rows are numbered in (batch, row) order.
#include <algorithm>
#include <map>
#include <new>
#include <string>
#include <tuple>

#include "edb_internal.h"

namespace {
using edb::fail;
constexpr int32_t UNSET = -1;

bool consecutive(const int32_t* s, int64_t n) {
    for (int64_t i = 0; i + 1 < n; ++i)
        if (s[i + 1] != s[i] + 1) return false;
    return true;
}

// Sort (key, value) pairs by their non-negative, distinct keys: LSD radix
// sort with 8-bit digits, as many passes as the largest key needs (a
// comparison sort for short lists).
void sort_by_key(std::vector<std::pair<int32_t, int32_t>>& a, std::vector<std::pair<int32_t, int32_t>>& tmp) {
    const size_t n = a.size();
    if (n < 64) {
        std::sort(a.begin(), a.end());
        return;
    }
    uint32_t maxk = 0;
    for (const auto& x : a) maxk = std::max(maxk, (uint32_t)x.first);
    tmp.resize(n);
    uint32_t count[256];
    for (int shift = 0; shift < 32 && (maxk >> shift) != 0; shift += 8) {
        std::fill(count, count + 256, 0u);
        for (const auto& x : a) ++count[((uint32_t)x.first >> shift) & 255u];
        uint32_t sum = 0;
        for (uint32_t& c : count) {
            const uint32_t t = c;
            c = sum;
            sum += t;
        }
        for (const auto& x : a) tmp[count[((uint32_t)x.first >> shift) & 255u]++] = x;
        a.swap(tmp);
    }
}
// PQ-tree layout (Section 3.2): slots from edb::pq_layout; each batch's rows
// follow the memory order of the first operand of its aligned group; an
// absent positional child reads its own zero pad.
void pq_descriptors(const edb_graph& g, const struct edb_schedule& s, const edb_operand_shape* shapes, edb_plan& pl,
                    const std::vector<int64_t>& idx_off, const std::vector<int64_t>& rag_off) {
    std::vector<int32_t> slot_of, lead;
    std::map<std::tuple<int, int, int>, int32_t> pad_of;
    edb::pq_layout(g, s, shapes, slot_of, pad_of, lead);
    const int32_t V = g.V, B = (int32_t)s.batch_type.size();
    const int32_t* bptr = s.batch_ptr.data();
    for (int32_t v = 0; v < V; ++v) pl.slot[v] = slot_of[v];
    for (const auto& kv : pad_of) pl.pads.push_back(slot_of[kv.second]);
    pl.n_slots = (int32_t)slot_of.size() + 1;
    std::vector<int32_t> list;
    std::vector<std::pair<int32_t, int32_t>> keyed;
    for (int32_t b = 0; b < B; ++b) {
        const edb_operand_shape& sh = shapes[s.batch_type[b]];
        const int32_t m = bptr[b + 1] - bptr[b];
        int32_t* ord = pl.order.data() + bptr[b];
        keyed.clear();
        for (int32_t r = 0; r < m; ++r) {
            const int32_t v = ord[r];
            int32_t key = slot_of[v];
            if (lead[b] > 0) {
                const int p = lead[b] - 1;
                const int32_t c = g.child_idx[g.child_ptr[v] + p];
                key = c >= 0 ? slot_of[c] : slot_of[pad_of.at({b, p, v})];
            }
            keyed.emplace_back(key, v);
        }
        std::sort(keyed.begin(), keyed.end());
        for (int32_t r = 0; r < m; ++r) ord[r] = keyed[r].second;
        int64_t off = idx_off[b] + m;
        edb_seg* sg = pl.segs.data() + pl.seg_ptr[b];
        const int nlists = sh.n_fixed + (sh.ragged ? 1 : 0);
        for (int li = 0; li < nlists; ++li) {
            list.clear();
            if (li < sh.n_fixed) {
                for (int32_t r = 0; r < m; ++r) {
                    const int32_t v = ord[r], c = g.child_idx[g.child_ptr[v] + li];
                    if (c >= 0) list.push_back(slot_of[c]);
                    else {
                        auto it = pad_of.find({b, li, v});
                        list.push_back(it == pad_of.end() ? -1 : slot_of[it->second]);
                    }
                }
            } else {
                int32_t* rp = pl.ragged_pool.data() + rag_off[b];
                rp[0] = 0;
                for (int32_t r = 0; r < m; ++r) {
                    const int32_t v = ord[r];
                    for (int64_t e = g.child_ptr[v] + sh.n_fixed; e < g.child_ptr[v + 1]; ++e)
                        if (g.child_idx[e] >= 0) list.push_back(slot_of[g.child_idx[e]]);
                    rp[r + 1] = (int32_t)list.size();
                }
            }
            edb_seg& q = sg[1 + li];
            const int64_t n = (int64_t)list.size();
            q.len = (int32_t)n;
            bool any = false;
            for (int32_t x : list) any |= x >= 0;
            if (li < sh.n_fixed) {
                // an all-absent positional list has no pads: no operand
                any = false;
                for (int32_t r = 0; r < m; ++r) any |= g.child_idx[g.child_ptr[ord[r]] + li] >= 0;
            }
            if (!any) {
                q.kind = EDB_SEG_NONE;
                q.idx_off = -1;
                continue;
            }
            int32_t* dst = pl.idx_pool.data() + off;
            for (int64_t e = 0; e < n; ++e) dst[e] = list[e] < 0 ? 0 : list[e];
            q.idx_off = off;
            q.base = dst[0];
            q.kind = consecutive(dst, n) ? EDB_SEG_CONTIG : EDB_SEG_GATHER;
            off += n;
        }
        int32_t* rs = pl.idx_pool.data() + idx_off[b];
        for (int32_t r = 0; r < m; ++r) rs[r] = slot_of[ord[r]];
        edb_seg& res = sg[0];
        res.idx_off = idx_off[b];
        res.len = m;
        res.base = m > 0 ? rs[0] : 0;
        res.kind = consecutive(rs, m) ? EDB_SEG_CONTIG : EDB_SEG_SCATTER;
    }
}
}  // namespace

extern "C" edb_status edb_plan_memory(const edb_graph_t* g, const edb_schedule_t* s,
                                      const edb_operand_shape* shapes, int32_t flags, edb_plan_t** out) {
    if (!out) return fail(EDB_ERR_INVALID, "edb_plan_memory: out is NULL");
    *out = nullptr;
    if (!g || !s || !shapes) return fail(EDB_ERR_INVALID, "edb_plan_memory: NULL argument");
    if (flags != EDB_PLAN_RC && flags != EDB_PLAN_IDENTITY && flags != EDB_PLAN_PQ)
        return fail(EDB_ERR_INVALID, "edb_plan_memory: unknown flags");
    if (s->V != g->V || s->T != g->T)
        return fail(EDB_ERR_INVALID, "edb_plan_memory: schedule does not belong to this graph");
    const int32_t V = g->V, T = g->T;
    for (int32_t t = 0; t < T; ++t)
        if (shapes[t].n_fixed < 0) return fail(EDB_ERR_INVALID, "edb_plan_memory: negative n_fixed");
    for (int32_t v = 0; v < V; ++v) {
        const edb_operand_shape& sh = shapes[g->op_type[v]];
        const int64_t cnt = g->child_ptr[v + 1] - g->child_ptr[v];
        if (cnt < sh.n_fixed || (!sh.ragged && cnt != sh.n_fixed))
            return fail(EDB_ERR_UNSUPPORTED, "edb_plan_memory: node " + std::to_string(v) +
                                                 " has " + std::to_string(cnt) + " children, its type expects " +
                                                 std::to_string(sh.n_fixed) + (sh.ragged ? "+" : ""));
        if (sh.has_x && g->x_row[v] < 0)
            return fail(EDB_ERR_INVALID, "edb_plan_memory: node " + std::to_string(v) + " has no x row");
    }
    edb_plan* p = new (std::nothrow) edb_plan;
    if (!p) return fail(EDB_ERR_OOM, "edb_plan_memory: out of host memory");
    try {
        const int32_t B = (int32_t)s->batch_type.size();
        const int32_t* bptr = s->batch_ptr.data();
        p->V = V;
        p->B = B;
        p->mode = flags;
        p->shapes.assign(shapes, shapes + T);
        p->slot.assign(V, UNSET);
        p->order.assign(s->batch_nodes.begin(), s->batch_nodes.end());
        int32_t* slot = p->slot.data();

        // layout of the descriptors, in ascending batch order:
        // segs: [result, positional lists..., ragged list] per batch
        // idx_pool: the slot list of every non-empty segment, same order
        // ragged_pool: m+1 row offsets per ragged batch
        std::vector<int64_t> idx_off(B + 1, 0), rag_off(B, -1);
        p->seg_ptr.assign(B + 1, 0);
        int64_t rag_total = 0;
        for (int32_t b = 0; b < B; ++b) {
            const edb_operand_shape& sh = shapes[s->batch_type[b]];
            const int32_t m = bptr[b + 1] - bptr[b];
            int64_t n = m + (int64_t)sh.n_fixed * m;
            if (sh.ragged) {
                int64_t rc = 0;
                for (int32_t i = bptr[b]; i < bptr[b + 1]; ++i) {
                    const int32_t v = s->batch_nodes[i];
                    for (int64_t e = g->child_ptr[v] + sh.n_fixed; e < g->child_ptr[v + 1]; ++e)
                        rc += g->child_idx[e] >= 0;
                }
                n += rc;
                rag_off[b] = rag_total;
                rag_total += m + 1;
            }
            idx_off[b + 1] = idx_off[b] + n;
            p->seg_ptr[b + 1] = p->seg_ptr[b] + 1 + sh.n_fixed + (sh.ragged ? 1 : 0);
        }
        p->idx_pool.assign((size_t)idx_off[B], 0);
        p->ragged_pool.assign((size_t)rag_total, 0);
        p->ragged_off.assign(rag_off.begin(), rag_off.end());
        p->segs.assign((size_t)p->seg_ptr[B], edb_seg{});

        if (flags == EDB_PLAN_PQ) {
            pq_descriptors(*g, *s, shapes, *p, idx_off, rag_off);
            goto x_rows;
        }
        {
        const bool identity = flags == EDB_PLAN_IDENTITY;
        int32_t next = 1;
        if (identity) {
            for (int32_t v = 0; v < V; ++v) slot[v] = v + 1;
            next = V + 1;
        }
        std::vector<int32_t> list, mark(V, -1);
        std::vector<std::pair<int32_t, int32_t>> setnodes, sort_tmp;
        int32_t stamp = 0;
        for (int32_t b = B - 1; b >= 0; --b) {
            const int32_t t = s->batch_type[b];
            const edb_operand_shape& sh = shapes[t];
            int32_t* ord = p->order.data() + bptr[b];
            const int32_t m = bptr[b + 1] - bptr[b];
            if (!identity) {
                // stable sort by slot, unset last: set nodes by slot, then unset in id order
                setnodes.clear();
                int32_t nu = 0;
                for (int32_t r = 0; r < m; ++r) {
                    if (slot[ord[r]] != UNSET) setnodes.emplace_back(slot[ord[r]], ord[r]);
                    else ord[nu++] = ord[r];   // compacts unset nodes to the front, order kept
                }
                if (!setnodes.empty()) {
                    sort_by_key(setnodes, sort_tmp);
                    const int32_t ns = (int32_t)setnodes.size();
                    for (int32_t r = nu - 1; r >= 0; --r) ord[r + ns] = ord[r];
                    for (int32_t r = 0; r < ns; ++r) ord[r] = setnodes[r].second;
                }
                for (int32_t r = 0; r < m; ++r)
                    if (slot[ord[r]] == UNSET) slot[ord[r]] = next++;
            }
            // operand lists, in order: positional children, then the ragged list
            int64_t off = idx_off[b] + m;
            edb_seg* sg = p->segs.data() + p->seg_ptr[b];
            const int nlists = sh.n_fixed + (sh.ragged ? 1 : 0);
            for (int li = 0; li < nlists; ++li) {
                list.clear();
                if (li < sh.n_fixed) {
                    for (int32_t r = 0; r < m; ++r) list.push_back(g->child_idx[g->child_ptr[ord[r]] + li]);
                } else {
                    int32_t* rp = p->ragged_pool.data() + rag_off[b];
                    rp[0] = 0;
                    for (int32_t r = 0; r < m; ++r) {
                        const int32_t v = ord[r];
                        for (int64_t e = g->child_ptr[v] + sh.n_fixed; e < g->child_ptr[v + 1]; ++e)
                            if (g->child_idx[e] >= 0) list.push_back(g->child_idx[e]);
                        rp[r + 1] = (int32_t)list.size();
                    }
                }
                const int64_t n = (int64_t)list.size();
                edb_seg& q = sg[1 + li];
                q.len = (int32_t)n;
                bool any = false, fresh = !identity;
                ++stamp;
                for (int32_t c : list) {
                    if (c < 0) continue;
                    any = true;
                    if (slot[c] != UNSET || mark[c] == stamp) fresh = false;
                    mark[c] = stamp;
                }
                if (!any) {
                    q.kind = EDB_SEG_NONE;
                    q.idx_off = -1;
                    continue;
                }
                int32_t* dst = p->idx_pool.data() + off;
                if (fresh) {
                    for (int64_t e = 0; e < n; ++e) {
                        if (list[e] < 0) p->pads.push_back(next);
                        else slot[list[e]] = next;
                        dst[e] = next++;
                    }
                } else {
                    for (int64_t e = 0; e < n; ++e) {
                        const int32_t c = list[e];
                        if (c >= 0 && slot[c] == UNSET) slot[c] = next++;
                        dst[e] = c >= 0 ? slot[c] : 0;
                    }
                }
                q.idx_off = off;
                q.base = dst[0];
                q.kind = (!identity && consecutive(dst, n)) ? EDB_SEG_CONTIG : EDB_SEG_GATHER;
                off += n;
            }
            // result list
            int32_t* rs = p->idx_pool.data() + idx_off[b];
            for (int32_t r = 0; r < m; ++r) rs[r] = slot[ord[r]];
            edb_seg& res = sg[0];
            res.idx_off = idx_off[b];
            res.len = m;
            res.base = m > 0 ? rs[0] : 0;
            res.kind = (!identity && consecutive(rs, m)) ? EDB_SEG_CONTIG : EDB_SEG_SCATTER;
        }
        p->n_slots = next;
        }

    x_rows:
        // x rows in (batch, row) order
        p->x_slot.assign(V, -1);
        int32_t nx = 0;
        for (int32_t b = 0; b < B; ++b) {
            if (!shapes[s->batch_type[b]].has_x) continue;
            for (int32_t i = bptr[b]; i < bptr[b + 1]; ++i) p->x_slot[p->order[i]] = nx++;
        }
    } catch (const std::bad_alloc&) {
        delete p;
        return fail(EDB_ERR_OOM, "edb_plan_memory: out of host memory");
    } catch (const std::exception& e) {
        delete p;
        return fail(EDB_ERR_INVALID, std::string("edb_plan_memory: internal error: ") + e.what());
    }
    edb::clear_error();
    *out = p;
    return EDB_OK;
}

extern "C" edb_status edb_plan_view(const edb_plan_t* p, edb_plan_view_t* v) {
    if (!p || !v) return fail(EDB_ERR_INVALID, "edb_plan_view: NULL argument");
    v->n_nodes = p->V;
    v->n_batches = p->B;
    v->n_slots = p->n_slots;
    v->n_pads = (int32_t)p->pads.size();
    v->slot = p->slot.data();
    v->order = p->order.data();
    v->x_slot = p->x_slot.data();
    v->seg_ptr = p->seg_ptr.data();
    v->segs = p->segs.data();
    v->idx_pool = p->idx_pool.data();
    v->idx_len = (int64_t)p->idx_pool.size();
    v->ragged_off = p->ragged_off.data();
    v->ragged_pool = p->ragged_pool.data();
    v->ragged_len = (int64_t)p->ragged_pool.size();
    v->pads = p->pads.data();
    return EDB_OK;
}

extern "C" void edb_plan_free(edb_plan_t* p) { delete p; }
