// Batching schedule: Algorithm 1 of ED-Batch (FSM-based dynamic batching) with
// a policy table keyed by the state encodings of Section 2.3, the agenda and
// depth heuristics of Section 2.1 as built-in policies, and the
// sufficient-condition heuristic (the type maximizing Eq. 1's frontier ratio,
// Lemma 1; Section 5's batch-count study).
//
// Frontier = unexecuted nodes whose present children have all executed.  Each
// step picks one type and batches every frontier node of that type, in
// ascending node id.  Ties go to the lowest type id; a table miss (or an
// action not on the frontier) falls back to the most common frontier type.
#include <algorithm>
#include <map>
#include <new>
#include <string>

#include "edb_internal.h"

namespace {

using edb::fail;

// Kahn order over present edges; depth(v) = 0 without present children,
// else 1 + max depth(child) (the input operation has depth 0).
void topo_depth(const edb_graph& g, std::vector<int64_t>& depth) {
    const int32_t V = g.V;
    std::vector<int32_t> pending(g.pending), queue;
    depth.assign(V, 0);
    queue.reserve(V);
    for (int32_t v = 0; v < V; ++v) if (pending[v] == 0) queue.push_back(v);
    for (size_t q = 0; q < queue.size(); ++q) {
        int32_t v = queue[q];
        for (int32_t i = g.cons_ptr[v]; i < g.cons_ptr[v + 1]; ++i) {
            int32_t p = g.cons[i];
            depth[p] = std::max(depth[p], depth[v] + 1);
            if (--pending[p] == 0) queue.push_back(p);
        }
    }
}

int32_t majority(const std::vector<int64_t>& counts) {
    int32_t best = -1;
    for (int32_t t = 0; t < (int32_t)counts.size(); ++t)
        if (counts[t] > 0 && (best < 0 || counts[t] > counts[best])) best = t;
    return best;
}

void encode(const std::vector<int64_t>& counts, int32_t enc, std::vector<int32_t>& key) {
    key.clear();
    for (int32_t t = 0; t < (int32_t)counts.size(); ++t)
        if (counts[t] > 0) key.push_back(t);
    if (enc == EDB_ENC_SORT) {
        std::stable_sort(key.begin(), key.end(),
                         [&](int32_t a, int32_t b) { return counts[a] > counts[b]; });
    } else if (enc == EDB_ENC_MAX) {
        key.push_back(majority(counts));
    }
}

}  // namespace

namespace edb {

void same_type_frontier(const edb_graph& g, std::vector<int32_t>& same_pending, std::vector<int64_t>& subf) {
    same_pending.assign(g.V, 0);
    subf.assign(g.T, 0);
    for (int32_t v = 0; v < g.V; ++v) {
        for (int64_t e = g.child_ptr[v]; e < g.child_ptr[v + 1]; ++e) {
            const int32_t c = g.child_idx[e];
            if (c >= 0 && g.op_type[c] == g.op_type[v]) ++same_pending[v];
        }
        if (same_pending[v] == 0) ++subf[g.op_type[v]];
    }
}

void same_type_executed(const edb_graph& g, int32_t v, std::vector<int32_t>& same_pending,
                        std::vector<int64_t>& subf) {
    const int32_t a = g.op_type[v];
    --subf[a];   // v was ready, so none of its children was pending
    for (int32_t i = g.cons_ptr[v]; i < g.cons_ptr[v + 1]; ++i) {
        const int32_t p = g.cons[i];
        if (g.op_type[p] == a && --same_pending[p] == 0) ++subf[a];
    }
}

int64_t lower_bound(const edb_graph& g) {
    // longest path, in nodes, of each type's induced subgraph, over a Kahn order
    std::vector<int32_t> pending(g.pending), queue, len(g.V, 1);
    std::vector<int64_t> best(g.T, 0);
    queue.reserve(g.V);
    for (int32_t v = 0; v < g.V; ++v) if (pending[v] == 0) queue.push_back(v);
    for (size_t q = 0; q < queue.size(); ++q) {
        const int32_t v = queue[q];
        best[g.op_type[v]] = std::max<int64_t>(best[g.op_type[v]], len[v]);
        for (int32_t i = g.cons_ptr[v]; i < g.cons_ptr[v + 1]; ++i) {
            const int32_t p = g.cons[i];
            if (g.op_type[p] == g.op_type[v]) len[p] = std::max(len[p], len[v] + 1);
            if (--pending[p] == 0) queue.push_back(p);
        }
    }
    int64_t total = 0;
    for (int64_t b : best) total += b;
    return total;
}

}  // namespace edb

extern "C" edb_status edb_lower_bound(const edb_graph_t* g, int64_t* lb) {
    if (!g || !lb) return fail(EDB_ERR_INVALID, "edb_lower_bound: NULL argument");
    try {
        *lb = edb::lower_bound(*g);
    } catch (const std::bad_alloc&) {
        return fail(EDB_ERR_OOM, "edb_lower_bound: out of host memory");
    }
    edb::clear_error();
    return EDB_OK;
}

extern "C" edb_status edb_schedule(const edb_graph_t* g, const edb_policy* pol, edb_schedule_t** out) {
    if (!out) return fail(EDB_ERR_INVALID, "edb_schedule: out is NULL");
    *out = nullptr;
    if (!g || !pol) return fail(EDB_ERR_INVALID, "edb_schedule: NULL graph or policy");
    if (pol->kind < EDB_POLICY_TABLE || pol->kind > EDB_POLICY_SUFFICIENT)
        return fail(EDB_ERR_INVALID, "edb_schedule: unknown policy kind");
    if (pol->kind == EDB_POLICY_TABLE && (pol->encoding < EDB_ENC_SORT || pol->encoding > EDB_ENC_MAX))
        return fail(EDB_ERR_INVALID, "edb_schedule: unknown state encoding");

    std::map<std::vector<int32_t>, int32_t> table;
    if (pol->kind == EDB_POLICY_TABLE && pol->table_len > 0) {
        if (!pol->table) return fail(EDB_ERR_TABLE, "edb_schedule: table is NULL with table_len > 0");
        const int32_t* f = pol->table;
        const int64_t L = pol->table_len;
        int64_t n = f[0], pos = 1;
        if (n < 0) return fail(EDB_ERR_TABLE, "edb_schedule: negative entry count");
        for (int64_t i = 0; i < n; ++i) {
            if (pos >= L) return fail(EDB_ERR_TABLE, "edb_schedule: table truncated");
            int64_t kl = f[pos];
            if (kl < 0 || pos + 1 + kl >= L) return fail(EDB_ERR_TABLE, "edb_schedule: bad key length");
            // a key naming a type outside [0, T) can never match a state
            std::vector<int32_t> key(f + pos + 1, f + pos + 1 + kl);
            table[key] = f[pos + 1 + kl];
            pos += 2 + kl;
        }
        if (pos != L) return fail(EDB_ERR_TABLE, "edb_schedule: trailing table entries");
    } else if (pol->kind == EDB_POLICY_TABLE && pol->table_len < 0) {
        return fail(EDB_ERR_TABLE, "edb_schedule: negative table_len");
    }

    struct edb_schedule* s = new (std::nothrow) struct edb_schedule;
    if (!s) return fail(EDB_ERR_OOM, "edb_schedule: out of host memory");
    try {
        const int32_t V = g->V, T = g->T;
        s->V = V;
        s->T = T;
        s->batch_ptr.push_back(0);
        s->batch_nodes.reserve(V);
        if (pol->kind == EDB_POLICY_DEPTH) {
            std::vector<int64_t> depth;
            topo_depth(*g, depth);
            std::vector<int32_t> ord(V);
            for (int32_t v = 0; v < V; ++v) ord[v] = v;
            std::stable_sort(ord.begin(), ord.end(), [&](int32_t a, int32_t b) {
                if (depth[a] != depth[b]) return depth[a] < depth[b];
                return g->op_type[a] < g->op_type[b];
            });
            for (int32_t i = 0; i < V; ++i) {
                int32_t v = ord[i];
                bool starts = i == 0 || depth[v] != depth[ord[i - 1]] || g->op_type[v] != g->op_type[ord[i - 1]];
                if (starts) {
                    if (i > 0) s->batch_ptr.push_back(i);
                    s->batch_type.push_back(g->op_type[v]);
                }
                s->batch_nodes.push_back(v);
            }
            if (V > 0) s->batch_ptr.push_back(V);
        } else {
            // pending counters and consumer lists over present edges (from ingest)
            std::vector<int32_t> pending(g->pending);
            const int32_t* cons_ptr = g->cons_ptr.data();
            const int32_t* cons = g->cons.data();
            const int32_t* op = g->op_type.data();
            // the ready nodes of each type as a bitmap over node ids (words
            // [lo, hi) may be non-zero): a batch comes out in ascending id by
            // scanning its type's words, without sorting
            const int64_t W = ((int64_t)V + 63) / 64;
            std::vector<uint64_t> ready((size_t)T * (size_t)W, 0);
            std::vector<int64_t> lo(T, W), hi(T, 0);
            std::vector<int64_t> counts(T, 0);
            auto make_ready = [&](int32_t v) {
                const int32_t a = op[v];
                const int64_t w = v >> 6;
                ready[(size_t)a * W + w] |= uint64_t(1) << (v & 63);
                lo[a] = std::min(lo[a], w);
                hi[a] = std::max(hi[a], w + 1);
                ++counts[a];
            };
            for (int32_t v = 0; v < V; ++v) if (pending[v] == 0) make_ready(v);
            std::vector<int64_t> depth, dsum(T, 0), dcnt(T, 0);
            if (pol->kind == EDB_POLICY_AGENDA) {
                topo_depth(*g, depth);
                for (int32_t v = 0; v < V; ++v) { dsum[op[v]] += depth[v]; dcnt[op[v]] += 1; }
            }
            // sufficient condition: sub-frontier of G^a = unexecuted type-a nodes
            // without an unexecuted type-a child (per edge occurrence)
            std::vector<int32_t> same_pending;
            std::vector<int64_t> subf;
            if (pol->kind == EDB_POLICY_SUFFICIENT) edb::same_type_frontier(*g, same_pending, subf);
            std::vector<int32_t> key;
            int64_t remaining = V;
            while (remaining > 0) {
                int32_t t = -1;
                if (pol->kind == EDB_POLICY_TABLE) {
                    encode(counts, pol->encoding, key);
                    auto it = table.find(key);
                    if (it != table.end()) t = it->second;
                    if (t < 0 || t >= T || counts[t] == 0) t = majority(counts);
                } else if (pol->kind == EDB_POLICY_SUFFICIENT) {
                    for (int32_t a = 0; a < T; ++a) {
                        if (counts[a] == 0) continue;
                        // |F_a(G)| / |F(G^a)| compared exactly, ties to the lowest id
                        if (t < 0 || counts[a] * subf[t] > counts[t] * subf[a]) t = a;
                    }
                } else {
                    for (int32_t a = 0; a < T; ++a) {
                        if (counts[a] == 0) continue;
                        // mean depth compared exactly: S_a * n_t < S_t * n_a
                        if (t < 0 || dsum[a] * dcnt[t] < dsum[t] * dcnt[a]) t = a;
                    }
                }
                if (t < 0) {
                    // nothing ready while nodes remain: a cycle (a graph built
                    // without the ingest's acyclicity check)
                    delete s;
                    return fail(EDB_ERR_CYCLE, "edb_schedule: the graph has a cycle");
                }
                // the batch: every node ready now, ascending; nodes that become
                // ready below wait for a later step
                const size_t first = s->batch_nodes.size();
                uint64_t* rw = ready.data() + (size_t)t * W;
                for (int64_t w = lo[t]; w < hi[t]; ++w) {
                    uint64_t x = rw[w];
                    rw[w] = 0;
                    while (x) {
                        s->batch_nodes.push_back((int32_t)(w * 64 + __builtin_ctzll(x)));
                        x &= x - 1;
                    }
                }
                lo[t] = W;
                hi[t] = 0;
                counts[t] = 0;
                const size_t last = s->batch_nodes.size();
                for (size_t i = first; i < last; ++i) {
                    const int32_t v = s->batch_nodes[i];
                    if (pol->kind == EDB_POLICY_AGENDA) { dsum[t] -= depth[v]; dcnt[t] -= 1; }
                    if (pol->kind == EDB_POLICY_SUFFICIENT) edb::same_type_executed(*g, v, same_pending, subf);
                    for (int32_t j = cons_ptr[v]; j < cons_ptr[v + 1]; ++j) {
                        const int32_t p = cons[j];
                        if (--pending[p] == 0) make_ready(p);
                    }
                }
                remaining -= (int64_t)(last - first);
                s->batch_ptr.push_back((int32_t)last);
                s->batch_type.push_back(t);
            }
        }
    } catch (const std::bad_alloc&) {
        delete s;
        return fail(EDB_ERR_OOM, "edb_schedule: out of host memory");
    }
    edb::clear_error();
    *out = s;
    return EDB_OK;
}

extern "C" edb_status edb_schedule_view(const edb_schedule_t* s, int32_t* n_batches,
                                        const int32_t** batch_ptr, const int32_t** batch_nodes,
                                        const int32_t** batch_type) {
    if (!s) return fail(EDB_ERR_INVALID, "edb_schedule_view: schedule is NULL");
    if (n_batches) *n_batches = (int32_t)s->batch_type.size();
    if (batch_ptr) *batch_ptr = s->batch_ptr.data();
    if (batch_nodes) *batch_nodes = s->batch_nodes.data();
    if (batch_type) *batch_type = s->batch_type.data();
    return EDB_OK;
}

extern "C" void edb_schedule_free(edb_schedule_t* s) { delete s; }
