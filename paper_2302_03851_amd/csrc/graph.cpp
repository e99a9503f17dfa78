// Typed dataflow graph ingest (Section 2.1 of ED-Batch: every operation carries
// a type; a mini-batch is the union of the per-instance graphs).
#include <new>
#include <string>

#include "edb_internal.h"

namespace edb {

static thread_local std::string g_last_error;

edb_status fail(edb_status st, const std::string& msg) {
    g_last_error = msg;
    return st;
}

void clear_error() { g_last_error.clear(); }

}  // namespace edb

extern "C" const char* edb_last_error(void) { return edb::g_last_error.c_str(); }

extern "C" int32_t edb_version(void) { return 10000; }

edb_status edb::build_graph(int32_t n_nodes, int32_t n_types, const int32_t* op_type, const int64_t* child_ptr,
                            const int32_t* child_idx, const int32_t* x_row, bool check_acyclic, edb_graph_t** out) {
    using edb::fail;
    if (!out) return fail(EDB_ERR_INVALID, "edb_build_graph: out is NULL");
    *out = nullptr;
    if (n_nodes < 0) return fail(EDB_ERR_INVALID, "edb_build_graph: n_nodes < 0");
    if (n_types < 1) return fail(EDB_ERR_INVALID, "edb_build_graph: n_types < 1");
    if (n_nodes > 0 && (!op_type || !child_ptr || !x_row))
        return fail(EDB_ERR_INVALID, "edb_build_graph: NULL array");
    if (n_nodes == 0 && !child_ptr) return fail(EDB_ERR_INVALID, "edb_build_graph: child_ptr is NULL");
    if (child_ptr[0] != 0) return fail(EDB_ERR_INVALID, "edb_build_graph: child_ptr[0] != 0");
    // monotone offsets first: every node's range then lies inside [0, E)
    for (int32_t v = 0; v < n_nodes; ++v)
        if (child_ptr[v + 1] < child_ptr[v])
            return fail(EDB_ERR_INVALID, "edb_build_graph: child_ptr not monotone at node " + std::to_string(v));
    const int64_t E = child_ptr[n_nodes];
    if (E > 0 && !child_idx) return fail(EDB_ERR_INVALID, "edb_build_graph: child_idx is NULL");
    edb_graph* g = new (std::nothrow) edb_graph;
    if (!g) return fail(EDB_ERR_OOM, "edb_build_graph: out of host memory");
    try {
        // one pass validates every node and counts, over present edges, each
        // node's children (pending) and each child's consumers (cons_ptr)
        std::vector<int32_t>& pend0 = g->pending;
        std::vector<int32_t>& cons_ptr = g->cons_ptr;
        std::vector<int32_t>& cons = g->cons;
        pend0.assign(n_nodes, 0);
        cons_ptr.assign(n_nodes + 1, 0);
        int32_t* pc = pend0.data();
        int32_t* cc = cons_ptr.data() + 1;
        std::string err;
        for (int32_t v = 0; v < n_nodes && err.empty(); ++v) {
            const int64_t e0 = child_ptr[v], e1 = child_ptr[v + 1];
            if (op_type[v] < 0 || op_type[v] >= n_types) { err = "op_type out of range at node "; err += std::to_string(v); break; }
            if (x_row[v] < -1) { err = "x_row < -1 at node "; err += std::to_string(v); break; }
            int32_t np = 0;
            for (int64_t e = e0; e < e1; ++e) {
                const int32_t c = child_idx[e];
                if (c < -1 || c >= n_nodes) { err = "child id out of range at node "; err += std::to_string(v); break; }
                if (c == v) { err = "self edge at node "; err += std::to_string(v); break; }
                if (c >= 0) { ++np; ++cc[c]; }
            }
            pc[v] = np;
        }
        if (!err.empty()) {
            delete g;
            return fail(EDB_ERR_INVALID, "edb_build_graph: " + err);
        }
        g->V = n_nodes;
        g->T = n_types;
        g->op_type.assign(op_type, op_type + n_nodes);
        g->child_ptr.assign(child_ptr, child_ptr + n_nodes + 1);
        g->child_idx.assign(child_idx, child_idx + E);
        g->x_row.assign(x_row, x_row + n_nodes);
        // consumers CSR over present edges
        for (int32_t v = 0; v < n_nodes; ++v) cons_ptr[v + 1] += cons_ptr[v];
        cons.resize(cons_ptr[n_nodes]);
        {
            std::vector<int32_t> fill(cons_ptr.begin(), cons_ptr.end() - 1);
            for (int32_t v = 0; v < n_nodes; ++v)
                for (int64_t e = child_ptr[v]; e < child_ptr[v + 1]; ++e)
                    if (child_idx[e] >= 0) cons[fill[child_idx[e]]++] = v;
        }
        if (check_acyclic) {
            // Kahn's algorithm: the graph must be acyclic
            std::vector<int32_t> pending(pend0), stack;
            stack.reserve(n_nodes);
            for (int32_t v = 0; v < n_nodes; ++v) if (pending[v] == 0) stack.push_back(v);
            int32_t seen = 0;
            while (!stack.empty()) {
                int32_t v = stack.back();
                stack.pop_back();
                ++seen;
                for (int32_t i = cons_ptr[v]; i < cons_ptr[v + 1]; ++i)
                    if (--pending[cons[i]] == 0) stack.push_back(cons[i]);
            }
            if (seen != n_nodes) {
                delete g;
                return fail(EDB_ERR_CYCLE, "edb_build_graph: the graph has a cycle");
            }
        }
    } catch (const std::bad_alloc&) {
        delete g;
        return fail(EDB_ERR_OOM, "edb_build_graph: out of host memory");
    }
    edb::clear_error();
    *out = g;
    return EDB_OK;
}

extern "C" edb_status edb_build_graph(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                                      const int64_t* child_ptr, const int32_t* child_idx,
                                      const int32_t* x_row, edb_graph_t** out) {
    return edb::build_graph(n_nodes, n_types, op_type, child_ptr, child_idx, x_row, true, out);
}

extern "C" void edb_graph_free(edb_graph_t* g) { delete g; }

extern "C" edb_status edb_graph_info(const edb_graph_t* g, int32_t* n_nodes, int32_t* n_types,
                                     int64_t* n_edges) {
    if (!g) return edb::fail(EDB_ERR_INVALID, "edb_graph_info: graph is NULL");
    if (n_nodes) *n_nodes = g->V;
    if (n_types) *n_types = g->T;
    if (n_edges) *n_edges = (int64_t)g->child_idx.size();
    return EDB_OK;
}
