// Internal structures shared by the host-side parts of the library.
#pragma once

#include <cstdint>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "edb.h"

struct edb_graph {
    int32_t V = 0, T = 0;
    std::vector<int32_t> op_type;
    std::vector<int64_t> child_ptr;
    std::vector<int32_t> child_idx;
    std::vector<int32_t> x_row;
    // consumers over present edges (CSR) and present-child counts, built once
    // during ingest and reused by every schedule
    std::vector<int32_t> cons_ptr, cons, pending;
};

struct edb_schedule {
    int32_t V = 0, T = 0;
    std::vector<int32_t> batch_ptr;    // [B+1]
    std::vector<int32_t> batch_nodes;  // [V]
    std::vector<int32_t> batch_type;   // [B]
};

struct edb_plan {
    int32_t V = 0, B = 0, n_slots = 0;
    std::vector<int32_t> slot, order, x_slot, seg_ptr, idx_pool, ragged_pool, pads;
    std::vector<int64_t> ragged_off;
    std::vector<edb_seg> segs;
    std::vector<edb_operand_shape> shapes;
    int32_t mode = EDB_PLAN_RC;
};

namespace edb {

// Thread-local last-error message; returns the status for `return fail(...)`.
edb_status fail(edb_status st, const std::string& msg);
void clear_error();

// edb_build_graph with the acyclicity check optional: without it the graph
// must go to a frontier policy's schedule, which reports a cycle itself (no
// node ready while some remain).
edb_status build_graph(int32_t n_nodes, int32_t n_types, const int32_t* op_type, const int64_t* child_ptr,
                       const int32_t* child_idx, const int32_t* x_row, bool check_acyclic, edb_graph_t** out);

// Sub-frontier bookkeeping for Eq. 1's ratio: same_pending[v] counts v's
// unexecuted present children of v's own type (per edge occurrence); subf[a]
// counts unexecuted type-a nodes with none, i.e. |Frontier(G^a)|.
void same_type_frontier(const edb_graph& g, std::vector<int32_t>& same_pending, std::vector<int64_t>& subf);
// Updates both after the ready node v executed.
void same_type_executed(const edb_graph& g, int32_t v, std::vector<int32_t>& same_pending,
                        std::vector<int64_t>& subf);
// Appendix A.3: sum over types of the longest path (in nodes) of the subgraph
// induced on that type.
int64_t lower_bound(const edb_graph& g);

// PQ-tree memory layout (Section 3.2): slot_of[x] for every variable (nodes,
// then one zero pad per absent entry of a positional list with a present
// entry), pad_of[(batch, child position, row node)] the pad variable, lead[b]
// the operand whose order batch b's rows follow (0 rows, 1 + p child p).
void pq_layout(const edb_graph& g, const struct edb_schedule& s, const edb_operand_shape* shapes,
               std::vector<int32_t>& slot_of, std::map<std::tuple<int, int, int>, int32_t>& pad_of,
               std::vector<int32_t>& lead);

// edb_forward's plain path (no executor handed back, no profiling): prepares
// the launches without device memory of their own, binds them to the device
// block cached for (current device, stream), copies the descriptors on the
// stream and launches (with use_graph through the stream's kept HIP graph of
// the same kernel sequence); the block grows in stream order when a call needs more.
edb_status forward_on_stream(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                             const edb_cell* cells, int32_t flags, const void* const* packed_weights,
                             const void* x, void* arena_h, void* arena_c, void* stream, bool use_graph);

}  // namespace edb
