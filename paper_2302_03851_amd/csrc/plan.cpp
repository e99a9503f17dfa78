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
// Slot 0 is the zero row.  x rows are numbered in (batch, row) order.
#include <algorithm>
#include <new>
#include <string>

#include "edb_internal.h"

namespace {
using edb::fail;
constexpr int32_t UNSET = -1;

bool consecutive(const int32_t* s, int64_t n) {
    for (int64_t i = 0; i + 1 < n; ++i)
        if (s[i + 1] != s[i] + 1) return false;
    return true;
}
}  // namespace

extern "C" edb_status edb_plan_memory(const edb_graph_t* g, const edb_schedule_t* s,
                                      const edb_operand_shape* shapes, int32_t flags, edb_plan_t** out) {
    if (!out) return fail(EDB_ERR_INVALID, "edb_plan_memory: out is NULL");
    *out = nullptr;
    if (!g || !s || !shapes) return fail(EDB_ERR_INVALID, "edb_plan_memory: NULL argument");
    if (flags != EDB_PLAN_RC && flags != EDB_PLAN_IDENTITY)
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
        p->V = V;
        p->B = B;
        p->mode = flags;
        p->shapes.assign(shapes, shapes + T);
        p->slot.assign(V, UNSET);
        p->order.assign(s->batch_nodes.begin(), s->batch_nodes.end());
        std::vector<int32_t>& slot = p->slot;
        // per batch, per list, per entry: the pad slot of an absent entry (fresh lists)
        std::vector<std::vector<std::vector<int32_t>>> pad_of(B);
        std::vector<std::vector<std::vector<int32_t>>> lists(B);
        std::vector<std::vector<int32_t>> rptr(B);

        auto build_lists = [&](int32_t b) {
            const int32_t t = s->batch_type[b];
            const edb_operand_shape& sh = shapes[t];
            const int32_t* ord = p->order.data() + s->batch_ptr[b];
            const int32_t m = s->batch_ptr[b + 1] - s->batch_ptr[b];
            auto& L = lists[b];
            L.assign(sh.n_fixed + (sh.ragged ? 1 : 0), {});
            for (int32_t q = 0; q < sh.n_fixed; ++q) {
                L[q].resize(m);
                for (int32_t r = 0; r < m; ++r) L[q][r] = g->child_idx[g->child_ptr[ord[r]] + q];
            }
            if (sh.ragged) {
                auto& R = L[sh.n_fixed];
                rptr[b].assign(1, 0);
                for (int32_t r = 0; r < m; ++r) {
                    const int32_t v = ord[r];
                    for (int64_t e = g->child_ptr[v] + sh.n_fixed; e < g->child_ptr[v + 1]; ++e)
                        if (g->child_idx[e] >= 0) R.push_back(g->child_idx[e]);
                    rptr[b].push_back((int32_t)R.size());
                }
            }
            pad_of[b].assign(L.size(), {});
        };

        int32_t next = 1;
        if (flags == EDB_PLAN_IDENTITY) {
            for (int32_t v = 0; v < V; ++v) slot[v] = v + 1;
            next = V + 1;
            for (int32_t b = 0; b < B; ++b) build_lists(b);
        } else {
            std::vector<int32_t> tmp;
            for (int32_t b = B - 1; b >= 0; --b) {
                int32_t* ord = p->order.data() + s->batch_ptr[b];
                const int32_t m = s->batch_ptr[b + 1] - s->batch_ptr[b];
                std::stable_sort(ord, ord + m, [&](int32_t a, int32_t c) {
                    const bool ua = slot[a] == UNSET, uc = slot[c] == UNSET;
                    if (ua != uc) return !ua;
                    return !ua && slot[a] < slot[c];
                });
                for (int32_t r = 0; r < m; ++r)
                    if (slot[ord[r]] == UNSET) slot[ord[r]] = next++;
                build_lists(b);
                for (size_t li = 0; li < lists[b].size(); ++li) {
                    const auto& L = lists[b][li];
                    bool any = false, fresh = true;
                    tmp.clear();
                    for (int32_t c : L) {
                        if (c < 0) continue;
                        any = true;
                        if (slot[c] != UNSET) fresh = false;
                        tmp.push_back(c);
                    }
                    if (!any) continue;
                    if (fresh) {
                        std::sort(tmp.begin(), tmp.end());
                        fresh = std::adjacent_find(tmp.begin(), tmp.end()) == tmp.end();
                    }
                    if (fresh) {
                        auto& pads = pad_of[b][li];
                        pads.assign(L.size(), 0);
                        for (size_t e = 0; e < L.size(); ++e) {
                            if (L[e] < 0) {
                                pads[e] = next;
                                p->pads.push_back(next);
                            } else {
                                slot[L[e]] = next;
                            }
                            ++next;
                        }
                    } else {
                        for (int32_t c : L)
                            if (c >= 0 && slot[c] == UNSET) slot[c] = next++;
                    }
                }
            }
        }
        for (int32_t v = 0; v < V; ++v)
            if (slot[v] == UNSET) {
                delete p;
                return fail(EDB_ERR_INVALID, "edb_plan_memory: node " + std::to_string(v) + " is not scheduled");
            }
        p->n_slots = next;

        // x rows in (batch, row) order
        p->x_slot.assign(V, -1);
        int32_t nx = 0;
        for (int32_t b = 0; b < B; ++b) {
            if (!shapes[s->batch_type[b]].has_x) continue;
            for (int32_t i = s->batch_ptr[b]; i < s->batch_ptr[b + 1]; ++i) p->x_slot[p->order[i]] = nx++;
        }

        // segment descriptors: result, positional lists, ragged list
        const bool indexed = flags == EDB_PLAN_IDENTITY;
        p->seg_ptr.push_back(0);
        p->ragged_off.assign(B, -1);
        std::vector<int32_t> ss;
        for (int32_t b = 0; b < B; ++b) {
            const int32_t* ord = p->order.data() + s->batch_ptr[b];
            const int32_t m = s->batch_ptr[b + 1] - s->batch_ptr[b];
            edb_seg res{};
            res.idx_off = (int64_t)p->idx_pool.size();
            res.len = m;
            for (int32_t r = 0; r < m; ++r) p->idx_pool.push_back(slot[ord[r]]);
            const int32_t* rs = p->idx_pool.data() + res.idx_off;
            res.kind = (!indexed && consecutive(rs, m)) ? EDB_SEG_CONTIG : EDB_SEG_SCATTER;
            res.base = rs[0];
            p->segs.push_back(res);
            for (size_t li = 0; li < lists[b].size(); ++li) {
                const auto& L = lists[b][li];
                edb_seg sg{};
                sg.len = (int32_t)L.size();
                bool any = false;
                for (int32_t c : L) any |= c >= 0;
                if (!any) {
                    sg.kind = EDB_SEG_NONE;
                    sg.idx_off = -1;
                    p->segs.push_back(sg);
                    continue;
                }
                sg.idx_off = (int64_t)p->idx_pool.size();
                const auto& pads = pad_of[b][li];
                for (size_t e = 0; e < L.size(); ++e)
                    p->idx_pool.push_back(L[e] >= 0 ? slot[L[e]] : (pads.empty() ? 0 : pads[e]));
                const int32_t* q = p->idx_pool.data() + sg.idx_off;
                sg.kind = (!indexed && consecutive(q, sg.len)) ? EDB_SEG_CONTIG : EDB_SEG_GATHER;
                sg.base = sg.len > 0 ? q[0] : 0;
                p->segs.push_back(sg);
            }
            p->seg_ptr.push_back((int32_t)p->segs.size());
            if (!rptr[b].empty()) {
                p->ragged_off[b] = (int64_t)p->ragged_pool.size();
                p->ragged_pool.insert(p->ragged_pool.end(), rptr[b].begin(), rptr[b].end());
            }
        }
    } catch (const std::bad_alloc&) {
        delete p;
        return fail(EDB_ERR_OOM, "edb_plan_memory: out of host memory");
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
