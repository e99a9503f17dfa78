// One call for one mini-batch: graph ingest, schedule, memory plan, launch
// preparation and asynchronous execution (the whole hot path, Algorithm 1 and
// Section 3.1 of ED-Batch), with every host object released before return.
// The call never waits for the GPU.  Without exec_out and EDB_PROFILE the
// launches use the device block the library keeps per device and stream
// (edb::forward_on_stream); otherwise an executor of their own, whose device
// buffers are freed in stream order after the work, and which can be handed
// back (exec_out) to read its launch records and, under EDB_PROFILE, the
// per-launch times.
#include <string>

#include "edb_internal.h"

extern "C" edb_status edb_forward(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                                  const int64_t* child_ptr, const int32_t* child_idx, const int32_t* x_row,
                                  const edb_policy* policy, const edb_operand_shape* shapes, int32_t plan_flags,
                                  const edb_cell* cells, int32_t exec_flags, const void* const* packed_weights,
                                  const void* x, void* arena_h, void* arena_c, int64_t arena_rows, void* stream,
                                  int32_t* n_slots, edb_exec_t** exec_out) {
    if (exec_out) *exec_out = nullptr;
    if (exec_flags & EDB_DRYRUN) return edb::fail(EDB_ERR_INVALID, "edb_forward: EDB_DRYRUN is not allowed");
    edb_graph_t* g = nullptr;
    edb_schedule_t* s = nullptr;
    edb_plan_t* p = nullptr;
    edb_exec_t* e = nullptr;
    // a frontier policy's schedule reports a cycle itself: the ingest skips its own check
    const bool frontier = policy && policy->kind != EDB_POLICY_DEPTH;
    edb_status st = edb::build_graph(n_nodes, n_types, op_type, child_ptr, child_idx, x_row, !frontier, &g);
    if (st == EDB_OK) st = edb_schedule(g, policy, &s);
    if (st == EDB_OK) st = edb_plan_memory(g, s, shapes, plan_flags, &p);
    if (st == EDB_OK) {
        if (n_slots) *n_slots = p->n_slots;
        if (arena_rows < p->n_slots)
            st = edb::fail(EDB_ERR_INVALID, "edb_forward: the arena has " + std::to_string(arena_rows) +
                                                " rows, the plan needs " + std::to_string(p->n_slots));
    }
    const bool use_graph = (exec_flags & EDB_USE_GRAPH) != 0;
    const int32_t flags = exec_flags & ~EDB_USE_GRAPH;
    if (st == EDB_OK && !exec_out && !(flags & EDB_PROFILE)) {
        // the plain path: the stream's cached device block, no per-call
        // allocation, upload stream, events or stream-ordered free
        st = edb::forward_on_stream(g, s, p, cells, flags, packed_weights, x, arena_h, arena_c, stream, use_graph);
    } else {
        if (st == EDB_OK) st = edb_prepare(g, s, p, cells, flags, &e);
        if (st == EDB_OK) st = edb_execute(e, packed_weights, x, arena_h, arena_c, stream);
    }
    // keep the error text of the failing step across the frees below
    const std::string err = st == EDB_OK ? std::string() : std::string(edb_last_error());
    if (st == EDB_OK && exec_out) *exec_out = e;
    else edb_exec_free(e);
    edb_plan_free(p);
    edb_schedule_free(s);
    edb_graph_free(g);
    if (st != EDB_OK) return edb::fail(st, err);
    return EDB_OK;
}
