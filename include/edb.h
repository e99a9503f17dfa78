/*
 * edb.h -- C ABI of the batched dynamic-dataflow-graph executor for AMD
 * MI355X (gfx950).
 *
 * The library executes the forward pass of a mini-batch of per-instance
 * dataflow graphs (chain LSTM, N-ary and child-sum TreeLSTM, lattice LSTM,
 * 2-D grid RNN) the way ED-Batch (arXiv 2302.03851) batches them:
 *
 *   edb_build_graph   typed graph ingest (Section 2.1: every operation has a
 *                     type; the mini-batch is the union of instance graphs)
 *   edb_schedule      Algorithm 1: repeatedly pick a type through a policy
 *                     table keyed by the frontier's state encoding
 *                     (Sections 2.2-2.3) and batch every ready node of it
 *   edb_plan_memory   batching-aware arena layout (Section 3.1: source and
 *                     result operands of a batch contiguous and aligned)
 *   edb_pack_weights  gate-interleaved weight layout for the fused cell kernels
 *   edb_prepare /     per batch one fused kernel on the GPU: operand gather ->
 *   edb_execute       cell GEMM on the matrix cores -> gate epilogue ->
 *                     scatter into the planned slots, the whole batch
 *                     sequence replayed from one HIP graph
 *
 * Conventions
 *   - Every call returns an edb_status.  On failure no output handle is
 *     created (*out is set to NULL) and edb_last_error() describes the error.
 *     No C++ exception crosses this interface.
 *   - Pointers documented as "host" are read during the call only; the
 *     library deep-copies what it keeps.  Pointers documented as "device"
 *     are caller-owned GPU memory the library never frees.
 *   - Handles are immutable after creation (except edb_exec_t, which caches
 *     its HIP graph) and may be read from several threads at once.
 */
#ifndef EDB_H
#define EDB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status ------------------------------------------------------------ */
typedef int32_t edb_status;
#define EDB_OK               0
#define EDB_ERR_INVALID     -1  /* bad argument: NULL, out of range, size mismatch */
#define EDB_ERR_CYCLE       -2  /* the graph is not a DAG */
#define EDB_ERR_OOM         -3  /* host or device allocation failed */
#define EDB_ERR_UNSUPPORTED -4  /* shape or cell configuration the kernels do not handle */
#define EDB_ERR_TABLE       -5  /* malformed policy table */
#define EDB_ERR_HIP         -6  /* a HIP runtime call failed (message holds the HIP error) */

/* Text of the last error on the calling thread; valid until the next call
 * into the library on that thread.  Never NULL. */
const char* edb_last_error(void);
/* Library version, major * 10000 + minor * 100 + patch. */
int32_t edb_version(void);

/* ---- graph (Section 2.1) ------------------------------------------------ */
typedef struct edb_graph edb_graph_t;

/* Typed dataflow graph in CSR form.
 *   n_nodes, n_types   V >= 0 nodes with types in [0, n_types), n_types >= 1
 *   op_type   host int32[V]      type of every node
 *   child_ptr host int64[V+1]    CSR offsets, child_ptr[0] == 0, non-decreasing
 *   child_idx host int32[E]      children of v: child_idx[child_ptr[v] .. child_ptr[v+1]);
 *                                positional children first, then ragged ones;
 *                                -1 = absent child (reads a zero state)
 *   x_row     host int32[V]      row of the caller's input matrix x holding v's
 *                                input vector, or -1 when v has none
 * Errors: EDB_ERR_INVALID for NULL arrays, ids out of range, a non-monotone
 * child_ptr or a self edge; EDB_ERR_CYCLE when the present edges contain a
 * cycle (checked with Kahn's algorithm). */
edb_status edb_build_graph(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                           const int64_t* child_ptr, const int32_t* child_idx,
                           const int32_t* x_row, edb_graph_t** out);
void edb_graph_free(edb_graph_t* g);
edb_status edb_graph_info(const edb_graph_t* g, int32_t* n_nodes, int32_t* n_types,
                          int64_t* n_edges);

/* ---- schedule (Algorithm 1, Sections 2.2-2.3) --------------------------- */
#define EDB_POLICY_TABLE  0  /* FSM policy table keyed by the state encoding */
#define EDB_POLICY_AGENDA 1  /* type of minimal mean topological depth (DyNet agenda) */
#define EDB_POLICY_DEPTH  2  /* groups of equal (depth, type) (TensorFlow Fold) */
#define EDB_POLICY_SUFFICIENT 3  /* type maximizing Eq. 1's frontier ratio (Lemma 1) */

#define EDB_ENC_SORT 0  /* frontier types sorted by frontier count desc, ties by id */
#define EDB_ENC_BASE 1  /* set of frontier types, ascending id */
#define EDB_ENC_MAX  2  /* E_base followed by the most common frontier type */

/* Batching policy.  `table` (host, may be NULL when table_len == 0) is a flat
 * int32 list [n_entries, {key_len, key[0..key_len), action} x n_entries]:
 * the state key (type ids in the encoding's order) maps to the next type.
 * A key that is missing, or an action that is not on the frontier, falls
 * back to the most common frontier type (ties to the lowest id).  Keys that
 * name types outside [0, n_types) never match.  A later entry with the same
 * key replaces an earlier one. */
typedef struct {
    int32_t kind;          /* EDB_POLICY_* */
    int32_t encoding;      /* EDB_ENC_* (table policy only) */
    const int32_t* table;  /* host */
    int64_t table_len;
} edb_policy;

typedef struct edb_schedule edb_schedule_t;

/* Runs the batching loop on the host.  Every batch holds all ready nodes of
 * the chosen type in ascending node id (Algorithm 1's frontier batch).
 * Errors: EDB_ERR_INVALID (NULL, unknown kind/encoding), EDB_ERR_TABLE;
 * EDB_ERR_CYCLE when no node is ready while nodes remain (the frontier
 * policies; only a graph with a cycle, which edb_build_graph rejects). */
edb_status edb_schedule(const edb_graph_t* g, const edb_policy* policy, edb_schedule_t** out);
/* Borrowed views, valid until edb_schedule_free:
 *   batch_ptr int32[n_batches+1], batch_nodes int32[V], batch_type int32[n_batches]. */
edb_status edb_schedule_view(const edb_schedule_t* s, int32_t* n_batches,
                             const int32_t** batch_ptr, const int32_t** batch_nodes,
                             const int32_t** batch_type);
void edb_schedule_free(edb_schedule_t* s);

/* Lower bound on the number of batches of any schedule (Appendix A.3): the
 * sum over types of the longest path, counted in nodes, of the subgraph
 * induced on that type's nodes (direct edges between them only).
 * Errors: EDB_ERR_INVALID (NULL). */
edb_status edb_lower_bound(const edb_graph_t* g, int64_t* lower_bound);

/* ---- learning the FSM policy (Section 2.3) ------------------------------ */
/* Tabular Q-learning with N-step bootstrapping over Algorithm 1's batching
 * loop.  State S_t = E(G_t) in the given encoding; actions = the frontier
 * types; reward (Eq. 1, its ratio taken as the worked example of Section 2.3
 * evaluates it, in (0, 1]):
 *     r = -1 + alpha * |Frontier_a(G_t)| / |Frontier(G^a_t)|
 * where G^a is the subgraph induced on type-a nodes.  The target of
 * Q(S_tau, a_tau) is the N-step return (gamma-discounted rewards of steps
 * tau .. tau+N-1, plus gamma^N max_a Q(S_{tau+N}, a) unless the episode ended
 * first), applied as Q += lr * (target - Q) as soon as S_{tau+N} is known,
 * and for the remaining steps, in order, when the episode ends.  Q starts at
 * 0.  Actions are epsilon-greedy; argmax ties go to the first action in the
 * state key.  Every check_every trials and after the last one the greedy
 * table (one entry per state with a Q entry) is scheduled; training stops
 * when that schedule reaches edb_lower_bound (Section 5.4 trains up to 1000
 * trials and checks every 50).  The learned table is that of the check with
 * the fewest batches, the earliest on ties.
 * Random draws: SplitMix64 (Steele, Lea and Flood 2014), draw k of the seed
 * being the finalizer of seed + (k+1) * 0x9E3779B97F4A7C15; training step c
 * (counted over all trials) explores when (draw 2c >> 11) * 2^-53 < epsilon and
 * then takes action number (draw 2c+1) mod (number of frontier types). */
typedef struct {
    int32_t encoding;     /* EDB_ENC_* */
    int32_t trials;       /* >= 1 (default 1000) */
    int32_t check_every;  /* >= 1 (default 50) */
    int32_t n_step;       /* N >= 1 (default 4) */
    double alpha;         /* > 0 (default 0.5) */
    double epsilon;       /* exploration probability in [0, 1] (default 0.1) */
    double lr;            /* learning rate in (0, 1] (default 0.2) */
    double gamma;         /* discount in [0, 1] (default 1) */
    uint64_t seed;        /* default 0 */
} edb_learn_params;

typedef struct {
    int32_t trials;       /* trials run */
    int32_t batches;      /* batches of the learned table's schedule */
    int64_t lower_bound;  /* edb_lower_bound of the graph */
    int32_t n_states;     /* entries of the learned table */
} edb_learn_stats;

typedef struct edb_learned edb_learned_t;

/* Fills *p with the defaults above. */
void edb_learn_defaults(edb_learn_params* p);
/* Learns a policy table for the graph (host only, single-threaded).
 * Errors: EDB_ERR_INVALID (NULL, parameters out of range), EDB_ERR_OOM. */
edb_status edb_learn_policy(const edb_graph_t* g, const edb_learn_params* p, edb_learned_t** out);
/* Borrowed view, valid until edb_learned_free: the table in edb_policy's flat
 * format (entries in ascending lexicographic key order) and the statistics. */
edb_status edb_learned_view(const edb_learned_t* l, const int32_t** table, int64_t* table_len,
                            edb_learn_stats* stats);
/* Borrowed view of the final Q function: n_states states in ascending key
 * order, keys flat as {key_len, key...} per state (keys_len int32 in all), and
 * q double[n_states * n_types] (0 for actions never updated). */
edb_status edb_learned_q(const edb_learned_t* l, int32_t* n_states, const int32_t** keys,
                         int64_t* keys_len, const double** q);
void edb_learned_free(edb_learned_t* l);

/* ---- memory plan (Section 3.1) ------------------------------------------ */
/* Operand shape of a type: exactly n_fixed positional children (-1 allowed),
 * then ragged children only when `ragged` is non-zero; has_x != 0 when the
 * type's cell reads an input row (then every node of it needs x_row >= 0). */
typedef struct {
    int32_t n_fixed;
    int32_t ragged;
    int32_t has_x;
} edb_operand_shape;

#define EDB_PLAN_RC       0  /* reverse consumer-first contiguous slot plan */
#define EDB_PLAN_IDENTITY 1  /* slot[v] = v + 1, every operand indexed (ablation) */
/* PQ-tree layout (Section 3.2, Algorithm 2): node states and one zero pad per
 * absent entry of a positional list with a present entry are ordered so that
 * as many batches as possible read and write contiguous, row-aligned
 * operands (PQ-tree reduction of every operand set, constraint broadcast
 * between a batch's operands, Q-node directions and P-node orders decided by
 * union-find).  A batch's rows follow the memory order of its first operand
 * that could be made consecutive.  Host cost grows with the batch sizes
 * (Lemma 2); ragged child lists only get adjacency, not alignment. */
#define EDB_PLAN_PQ       2

#define EDB_SEG_NONE    0  /* operand absent in every row: nothing to load */
#define EDB_SEG_CONTIG  1  /* rows base, base+1, ... */
#define EDB_SEG_GATHER  2  /* source rows listed in the index pool */
#define EDB_SEG_SCATTER 3  /* result rows listed in the index pool */

/* One operand list of a batch.  Rows are slot numbers of the node-state
 * arena (slot 0 is the all-zero row; pad slots are zero and never written). */
typedef struct {
    int32_t kind;     /* EDB_SEG_* */
    int32_t base;     /* CONTIG: first slot */
    int64_t idx_off;  /* GATHER/SCATTER: offset of the slot list in idx_pool */
    int32_t len;      /* number of entries (rows) */
    int32_t reserved;
} edb_seg;

typedef struct edb_plan edb_plan_t;

/* Plan the arena.  shapes: host [n_types].  Segment layout per batch b:
 * segs[seg_ptr[b]] is the result list (CONTIG or SCATTER), followed by one
 * source list per positional child, followed by the ragged list when the
 * type is ragged.  Ragged lists hold only present children; ragged_ptr gives
 * each row's entries.
 * Errors: EDB_ERR_INVALID (NULL, flags, a node of a has_x type without x),
 * EDB_ERR_UNSUPPORTED (a node's child count does not fit its type's shape). */
edb_status edb_plan_memory(const edb_graph_t* g, const edb_schedule_t* s,
                           const edb_operand_shape* shapes, int32_t flags, edb_plan_t** out);

typedef struct {
    int32_t n_nodes, n_batches, n_slots, n_pads;
    const int32_t* slot;        /* [V] arena row of each node */
    const int32_t* order;       /* [V] rows of batch b: order[batch_ptr[b] .. batch_ptr[b+1]) */
    const int32_t* x_slot;      /* [V] row of the node's input in the staged x buffer, -1 if none */
    const int32_t* seg_ptr;     /* [n_batches+1] */
    const edb_seg* segs;        /* [seg_ptr[n_batches]] */
    const int32_t* idx_pool;    /* [idx_len] */
    int64_t idx_len;
    const int64_t* ragged_off;  /* [n_batches] offset of the batch's m+1 row offsets in ragged_pool, -1 if none */
    const int32_t* ragged_pool;
    int64_t ragged_len;
    const int32_t* pads;        /* [n_pads] pad slots */
} edb_plan_view_t;

/* Borrowed view, valid until edb_plan_free. */
edb_status edb_plan_view(const edb_plan_t* p, edb_plan_view_t* view);
void edb_plan_free(edb_plan_t* p);

/* ---- cells and weights ---------------------------------------------------- */
#define EDB_CELL_LSTM_CHAIN    0  /* children [prev];            gates [i,f,g,o]          */
#define EDB_CELL_NARY_LEAF     1  /* no children, x;             gates [i,o,u]            */
#define EDB_CELL_NARY_INTERNAL 2  /* children [h_0, h_1], no x;  gates [i,f_0,f_1,o,u]    */
#define EDB_CELL_GRID          3  /* children [left, top], x;    gates [i,f_l,f_t,o,u]    */
#define EDB_CELL_CS_LEAF       4  /* no children, x;             gates [i,o,u]            */
#define EDB_CELL_CS_INTERNAL   5  /* ragged children, no x;      [i,o,u] on sum h, f per child */
#define EDB_CELL_LAT_CHAR      6  /* [prev char] + ragged words; gates [i,f,o,u] + link gates */
#define EDB_CELL_LAT_WORD      7  /* [first char], x;            gates [i,f,u], no h output */
/* TreeGRU (Table 2): the gated recurrent unit over two ordered children, the
 * reset gates applied after the recurrent products.  A GRU node's state is
 * written to both arenas (h and, in fp32, c); children's states are read from
 * the c arena.  Leaf: h = (1 - sigma(z)) tanh(n).  Internal:
 * h = sigma(z) (h_0 + h_1) / 2 + (1 - sigma(z)) tanh(sigma(r_0) n_0 + sigma(r_1) n_1). */
#define EDB_CELL_GRU_LEAF      8  /* no children, x;             gates [z,n]              */
#define EDB_CELL_GRU_INTERNAL  9  /* children [h_0, h_1], no x;  gates [z,r_0,r_1,n_0,n_1] */
/* MV-RNN (Table 2; every tree node carries a vector and a d x d matrix, d =
 * hidden).  A node's matrix is held as d graph nodes, node j = column j of
 * the matrix, so that every state is a row of the arena.  An internal tree
 * node with left child (a, A) and right child (b, B) has vector
 * tanh(W [B a ; A b] + b_W) and matrix W_M [A ; B].  All three kinds write h
 * and (fp32) the same values to c.
 *   LINEAR: h = x W + b (a leaf's vector and matrix columns, W the identity).
 *   MV_MAT: children [column j of A, column j of B]; h = [h_0, h_1] W + b
 *           (W = W_M transposed).
 *   MV_VEC: children [a, b], then exactly 2H more: the H column nodes of A,
 *           then the H column nodes of B; h = tanh([B a, A b] W + b) (W = the
 *           model's W transposed).  B a = sum_j a_j (column j of B) is
 *           computed by a launch of its own before the GEMM.
 * The three MV-RNN kinds run in fp32 only (EDB_ERR_UNSUPPORTED for bf16). */
#define EDB_CELL_LINEAR       10  /* no children, x;             h = x W + b              */
#define EDB_CELL_MV_MAT       11  /* children [h_0, h_1], no x;  h = [h_0, h_1] W + b     */
#define EDB_CELL_MV_VEC       12  /* children [a, b] + 2H matrix columns; tanh            */
/* Lattice GRU (Table 2): every incoming edge of a lattice position proposes a
 * GRU step (reset gate after the recurrent product) from its source position's
 * state with its own input; the position's state is the mean of the
 * proposals.  Both kinds write h and (fp32) the same values to c; the edge
 * reads its source's state from the c arena.  fp32 only.
 *   LGRU_EDGE: child [source position], x; gates [z, r, n_x, n_h];
 *              h = (1 - sigma(z)) n + sigma(z) h_src, n = tanh(n_x + sigma(r) n_h).
 *   POOL_MEAN: ragged children (the edges), no x; h = (mean of their h) W + b
 *              (W the identity and b = 0 for the plain mean; no edge: h = b). */
#define EDB_CELL_LGRU_EDGE    13  /* [source], x;                gates [z,r,n_x,n_h]      */
#define EDB_CELL_POOL_MEAN    14  /* ragged children, no x;      mean of their h, then W  */

#define EDB_F32  0  /* W, x, h fp32 */
#define EDB_BF16 1  /* W, x, h bf16 (round to nearest even); c fp32; fp32 accumulation */

typedef struct {
    int32_t kind;        /* EDB_CELL_* */
    int32_t in_dim;      /* E (ignored by kinds without x) */
    int32_t hidden;      /* H, equal for every type of a graph */
    int32_t n_children;  /* N of NARY_INTERNAL (only 2 is supported); 0 otherwise */
    int32_t dtype;       /* EDB_F32 or EDB_BF16 */
} edb_cell;

/* Bytes of the packed weight buffer of one cell type. */
edb_status edb_packed_weight_bytes(const edb_cell* cell, int64_t* bytes);

/* Pack the logical weights of one cell type into the gate-interleaved,
 * zero-padded device layout the kernels read.  (Section 3, static subgraphs,
 * and the discussion of Table 3: the gates of one cell run as one batched
 * operation over one weight operand, the cell is a static subgraph whose
 * operators are batched together; here all gates of a hidden unit block sit
 * in one contiguous weight block so that one GEMM computes every gate.)  `logical` is a host array of
 * float32 row-major matrices in this order (K x N, rows [x ; child h ...],
 * columns gate-major in the kind's gate order):
 *   LSTM_CHAIN     W[(E+H) x 4H], b[4H]
 *   NARY_LEAF      W[E x 3H], b[3H]          (CS_LEAF alike)
 *   NARY_INTERNAL  U[2H x 5H], b[5H]
 *   GRID           W[(E+2H) x 5H], b[5H]
 *   CS_INTERNAL    U_iou[H x 3H], U_f[H x H], b_iou[3H], b_f[H]
 *   LAT_WORD       W[(E+H) x 3H], b[3H]
 *   LAT_CHAR       W[(E+H) x 4H], W_lx[E x H], W_lc[H x H], b[4H], b_l[H]
 *   GRU_LEAF       W[E x 2H], b[2H]
 *   GRU_INTERNAL   U[2H x 5H], b[5H]   (the n_0 columns use child 0's rows only,
 *                                       the n_1 columns child 1's; the other
 *                                       blocks of those columns are ignored)
 *   LINEAR         W[E x H], b[H]
 *   MV_MAT         W[2H x H], b[H]     (rows: child 0's column, then child 1's)
 *   MV_VEC         W[2H x H], b[H]     (rows: B a, then A b)
 *   LGRU_EDGE      W[(E+H) x 4H], b[4H] (n_x's columns use the x rows only, n_h's
 *                                       the source rows only; b of n_h = b_hn)
 *   POOL_MEAN      W[H x H], b[H]
 * bf16 cells round the matrices to bf16 (ties to even); biases stay fp32.
 * packed_dev: device buffer of edb_packed_weight_bytes bytes (caller-owned).
 * The copy is enqueued on `stream` (hipStream_t, NULL = default stream) and
 * has completed when the call returns. */
edb_status edb_pack_weights(const edb_cell* cell, const float* const* logical,
                            void* packed_dev, void* stream);

/* ---- execution ------------------------------------------------------------ */
#define EDB_USE_GRAPH    1  /* run the batch sequence as one HIP graph launch (graph kept per stream) */
#define EDB_DRYRUN       2  /* record the launch list only; no HIP call (CPU testing) */
#define EDB_FORCE_GATHER 4  /* treat every CONTIG operand as indexed (ablation) */
#define EDB_X_DIRECT     8  /* read x rows in place by x_row instead of staging them */
#define EDB_PROFILE     16  /* eager launches timed by start/stop HIP events in each dispatch (edb_exec_launch_times) */
#define EDB_NO_FLOW     32  /* one launch per batch only (no dataflow launches) */
#define EDB_NO_SPLIT_K  64  /* small tiles without split-K only (each accumulator sums its k-groups in order) */
#define EDB_TILE_LARGE 128  /* the large bf16 tile for every batch it supports, whatever the batch size */
#define EDB_NO_LARGE   256  /* never the large tile (ablation) */
#define EDB_FLOW_DRYRUN 512 /* with EDB_DRYRUN only: build the dataflow launches (switched off on the
                               GPU) so that edb_exec_validate can check their descriptors */

typedef struct edb_exec edb_exec_t;

/* Bind a graph, schedule and plan to cell kernels.  cells: host [n_types].
 * (Section 3.1: each batch of the schedule (Algorithm 1) becomes one batched
 * operation whose source operands are gathered and whose results are
 * scattered according to the memory plan; this call turns the plan's operand
 * lists into the device descriptors that the fused kernels read, so that the
 * gather and scatter happen inside the batch's kernel.)
 * Uploads the batch descriptors and index lists to the current HIP device
 * and allocates the staged-x buffer; both are owned by the handle.
 * Each batch gets the tile variant of smallest estimated time: small tiles
 * (16-32 rows per work-group, the operand rows staged in LDS, optional
 * split-K over the waves), streamed tiles (the same shapes for kinds without
 * a ragged phase, every lane loading its own operand fragments) for the many
 * small batches, the large bf16 tile (64-256 rows, both operands through LDS)
 * for batches of thousands of rows, and for bf16 x-only leaf batches of at
 * least 8192 rows the weight-stationary tile (32 units' weights held in LDS for
 * the whole launch, 256-row tiles walked in turn; off under EDB_NO_LARGE and
 * when another variant is forced).  Without split-K (EDB_NO_SPLIT_K, and
 * always in the large and weight-stationary tiles) a batch's results do not
 * depend on the variant:
 * they are bitwise equal across variants, layouts and launch modes; with it,
 * variants with the same reduction split (a streamed tile and its staged
 * counterpart) are bitwise equal.  For sweeps and tests, the environment
 * variable EDB_VARIANT=v (read at each call) forces variant v on every batch
 * whose cell kind has it; a forced streamed variant falls back to its staged
 * counterpart on the other kinds.
 * Errors: EDB_ERR_INVALID, EDB_ERR_UNSUPPORTED (dimension or kind mix the
 * kernels do not handle), EDB_ERR_OOM, EDB_ERR_HIP. */
edb_status edb_prepare(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                       const edb_cell* cells, int32_t flags, edb_exec_t** out);

/* Run one forward pass, asynchronously on `stream` (hipStream_t): the batches
 * in the order Algorithm 1 produced them, each as one launch of its fused
 * gather / cell GEMM / gate epilogue / scatter kernel (Section 3.1); with
 * EDB_USE_GRAPH the whole sequence is one graph launch (Section 1: fewer
 * kernel launches is the first reason batching pays).
 *   packed_weights host array [n_types] of device pointers (edb_pack_weights output)
 *   x        device [n_x_rows x in_dim] of the cells' dtype, rows addressed by x_row
 *   arena_h  device [n_slots x H] of the cells' dtype; node v's h is row slot[v]
 *   arena_c  device [n_slots x H] fp32;               node v's c is row slot[v]
 * The call zeroes the arena's zero row and pad rows, stages x, then runs
 * every batch in schedule order.  x is not staged under EDB_X_DIRECT, when
 * every node's staged row would be its own row of x (x is then read in
 * place), or when a single batch reads x (it then reads the caller's rows
 * through its row list, as under EDB_X_DIRECT).  With
 * EDB_USE_GRAPH the sequence runs as one launch of a HIP graph that the
 * library keeps per device and stream and reuses for every later execution
 * there, of any executor, whose sequence has the same kernels and block sizes
 * (a new input graph of the same shape of schedule): the graph's kernel nodes
 * get the new arguments, grids and LDS sizes in place, without a new
 * instantiation; up to 4 sequences per stream are kept, the least recently
 * used one replaced (after its last launch has run); they live until
 * edb_stream_release on the stream or the end of the process.  Kernel faults surface at the caller's next synchronisation.
 * One edb_exec_t must not run on two streams at once. */
edb_status edb_execute(edb_exec_t* e, const void* const* packed_weights, const void* x,
                       void* arena_h, void* arena_c, void* stream);

/* Graph reuse counters of the process (EDB_USE_GRAPH executions): the kernel
 * sequences instantiated as new HIP graphs, and the executions that instead
 * updated the nodes of a kept graph in place (Section 1 prices a launch;
 * dynamic inputs change the graph every mini-batch, so a new input must not
 * cost a new instantiation).  Host outputs; EDB_ERR_INVALID on NULL. */
edb_status edb_graph_stats(int64_t* instantiated, int64_t* updated);

/* Dataflow launches (a persistent kernel running a run of consecutive small
 * batches, each tile waiting only for the tiles that produce its operand
 * rows) are currently switched off: every batch runs as its own launch and
 * EDB_NO_FLOW has no effect.  edb_exec_check reports a timed-out dataflow
 * wait when they are enabled.
 *
 * Number of launch records of one edb_execute: record 0 is the staging launch
 * (x staging and the clearing of the zero and pad rows), then the batches'
 * launches.  Record 0 has grid 0 and is not issued when nothing is staged and
 * the first batch (no child lists, no x padding) clears those rows itself. */
edb_status edb_exec_launches(const edb_exec_t* e, int32_t* n_kernels);

/* Description of launch i (for tests and profiling). */
typedef struct {
    int32_t batch;     /* batch index (first batch of a dataflow launch), -1 for the staging kernel */
    int32_t kind;      /* EDB_CELL_* of the batch, -1 for staging and dataflow launches */
    int32_t m;         /* rows (all batches of a dataflow launch) */
    int32_t k;         /* padded reduction length of the main GEMM */
    int32_t n;         /* padded output columns (gates x padded hidden) */
    int32_t variant;   /* tile variant id: 0-7 small tiles, 8-10 and 15-16 the large tile (size
                          classes 0-4: 256, 128, 64 rows x 64 units, then 64 and 32 rows x 32
                          units, fewer rows for 5-gate cells), 11-14 streamed tiles (counterparts
                          of the small tiles 3, 6, 4, 5), 17 the weight-stationary tile
                          (256-row tiles x 32 units, 512 threads), 100 a dataflow launch */
    int32_t grid;      /* work-groups */
    int32_t block;     /* threads per work-group */
    int32_t seg_kind[4]; /* kinds of result, child 0, child 1, ragged lists */
    int32_t n_batches; /* batches the launch executes (0 for staging and for parts 1, 2) */
    int32_t part;      /* 0: the batch's cell kernel.  A child-sum batch on the large tile runs
                          as three launches in this order: 2 the forget GEMM over its children
                          (m = children), 1 per parent the child sum of h and the sum of the
                          children's sigma(f_k) c_k, then 0 the parents.  An MV_VEC batch runs
                          as 1 the matrix-vector products [B a, A b], then 0 its GEMM */
} edb_launch_info;
edb_status edb_exec_launch_info(const edb_exec_t* e, int32_t i, edb_launch_info* info);

/* Per-launch GPU durations of the last edb_execute of an EDB_PROFILE handle,
 * in milliseconds: each kernel's own duration, from start and stop HIP events
 * that the dispatch packet records on the execution stream (0 for a record
 * with grid 0, which is not issued).  ms: host float[n], n = edb_exec_launches.
 * Waits for that execution to finish.  EDB_ERR_INVALID without EDB_PROFILE
 * or before the first execute. */
edb_status edb_exec_launch_times(edb_exec_t* e, float* ms, int32_t n);

/* The whole path for one mini-batch in one call (Section 2.1: a mini-batch
 * is the union of per-instance dataflow graphs; Algorithm 1 batches it and
 * Section 3 lays out its memory, all at run time for every new input):
 * edb_build_graph, edb_schedule, edb_plan_memory, edb_prepare (eager
 * launches) and edb_execute on `stream`, then every handle is released.  The call does not
 * wait for the GPU.  Device memory: without exec_out and EDB_PROFILE the call
 * uses a device block that the library keeps for the current device and
 * `stream` and reuses on the next call there (the descriptors are copied on
 * `stream` from pinned host buffers of a pool that the library keeps for the
 * process, so the next call overwrites them after this call's kernels); the
 * block grows in stream order when a call needs more (EDB_ERR_OOM if it
 * cannot) and is held until edb_stream_release.  Calls on one stream from
 * several threads enqueue one at a time.  With exec_out or EDB_PROFILE the
 * executor has device buffers of its own, freed in stream order after the
 * work.  Arguments are those of the individual calls; arena_h and
 * arena_c must hold at least the plan's n_slots rows (arena_rows), which is
 * returned in *n_slots (may be NULL) also when the arena is too small
 * (EDB_ERR_INVALID).  EDB_DRYRUN is rejected.  EDB_USE_GRAPH (plain path:
 * no exec_out, no EDB_PROFILE) runs the launches through the stream's kept
 * graph as edb_execute does.  With a frontier policy the
 * ingest leaves the acyclicity check to the schedule, which returns
 * EDB_ERR_CYCLE for a cycle as edb_build_graph would.
 * exec_out (may be NULL): on success receives the executor instead of it
 * being freed; the caller reads edb_exec_launch_info and, with EDB_PROFILE in
 * exec_flags, edb_exec_launch_times, and releases it with edb_exec_free. */
edb_status edb_forward(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                       const int64_t* child_ptr, const int32_t* child_idx, const int32_t* x_row,
                       const edb_policy* policy, const edb_operand_shape* shapes, int32_t plan_flags,
                       const edb_cell* cells, int32_t exec_flags, const void* const* packed_weights,
                       const void* x, void* arena_h, void* arena_c, int64_t arena_rows, void* stream,
                       int32_t* n_slots, edb_exec_t** exec_out);

/* Returns the device block that edb_forward keeps for the current device
 * and `stream` (a stream-ordered free on `stream`, after the work already
 * enqueued there; the call waits for the copies of the stream's descriptors
 * to have run); a later edb_forward on the stream allocates a new one.  The
 * pinned host memory of the copies comes from a pool that the library keeps
 * for the life of the process.  The HIP graphs kept for the stream
 * (EDB_USE_GRAPH) are destroyed too, each after its last launch has run.
 * Call it before destroying a stream that edb_forward or an EDB_USE_GRAPH
 * execution used, and not while another thread enqueues work on it.  No
 * block and no graph: a no-op.  Errors: EDB_ERR_HIP. */
edb_status edb_stream_release(void* stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): edb_forward without any
 * device allocation.  The executor's device memory (batch descriptors and
 * index lists, staged x, the child-sum and MV-RNN scratch rows) lives in one
 * fixed array of EDB_NOALLOC_SCRATCH_BYTES bytes per device, which the
 * library's code object holds on every device it runs on until the process
 * ends; its address is looked up once per device on the first call there.
 * The descriptors are copied to it on `stream` (from host memory that the
 * call reads before returning) and every kernel runs eagerly on `stream`.
 * Arguments and results are those of edb_forward (no executor is handed
 * back); EDB_USE_GRAPH, EDB_PROFILE and EDB_DRYRUN are rejected
 * (EDB_ERR_INVALID).  A mini-batch whose device memory exceeds the array is
 * rejected with EDB_ERR_UNSUPPORTED before anything is enqueued.  The call
 * makes no hipMalloc, hipFree, stream or event creation.  Every call on a
 * device shares that device's array and the array keeps the last call's
 * contents: calls on one device must be ordered (the same stream, or streams
 * the caller synchronises); calls that overlap on one device race. */
#define EDB_NOALLOC_SCRATCH_BYTES (32LL << 20)
edb_status edb_forward_noalloc(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                               const int64_t* child_ptr, const int32_t* child_idx, const int32_t* x_row,
                               const edb_policy* policy, const edb_operand_shape* shapes, int32_t plan_flags,
                               const edb_cell* cells, int32_t exec_flags, const void* const* packed_weights,
                               const void* x, void* arena_h, void* arena_c, int64_t arena_rows, void* stream,
                               int32_t* n_slots);

/* Host-side check of an executor's device descriptors (works on EDB_DRYRUN
 * handles; no HIP call).  The int buffer that edb_prepare uploads is decoded
 * the way the kernels read it: every launch's operand lists (positional,
 * ragged, x and result lists, ragged offsets) and, for a dataflow launch, its
 * batch descriptors, tile records, dependency ranges and counter offsets.
 * Every read is bounds-checked; the forward pass is replayed at the level of
 * arena rows (each result slot written once, never the zero row or a pad,
 * every row read after the launch or the dataflow row tile that writes it,
 * which must be among the reading row tile's dependencies and hold smaller
 * tickets), and each dataflow launch's ticket and dependency protocol is
 * emulated with min(n_workers, grid) work-groups in several interleavings.
 * *checked (may be NULL): launches and dataflow row tiles checked.
 * EDB_ERR_INVALID with the first problem found in edb_last_error(). */
edb_status edb_exec_validate(const edb_exec_t* e, int32_t n_workers, int64_t* checked);

/* Wait for `stream` and check the last execution's dataflow launches:
 * EDB_ERR_HIP if a bounded wait timed out (the results are then invalid). */
edb_status edb_exec_check(edb_exec_t* e, void* stream);

/* ---- Diagnostics: split-phase copies and roofline probes ---- */

/* Split-phase diagnostic.  Section 3.1 prices a batch as a gather of its
 * operand rows into one contiguous buffer, the batched computation, and a
 * scatter of the results to their consumers' slots; the fused kernels of
 * edb_execute do both copies inside the cell kernel.  edb_split_phase runs
 * them alone, batch by batch in schedule order, on `stream`:
 *   gather:  the rows the batch's cell kernel reads (x rows of the x the
 *            executor reads; for each positional and each ragged child entry
 *            its h row and its c row, absent children as the zero row) are
 *            copied into `buf`, densely, one list after the other;
 *   scatter: m rows of h and m rows of c are copied from the start of `buf`
 *            into the batch's result slots.
 * No cell is computed: afterwards the arenas hold copied rows, not states
 * (run edb_execute again for states).  The executor must have run
 * (edb_execute stages x).  buf: device, 16-byte aligned, at least
 * edb_split_phase_bytes bytes (the largest batch's dense lists).
 * ms (may be NULL): host float[n], n >= 2 * n_batches; receives per batch the
 * gather and the scatter kernel's duration in milliseconds (HIP events in the
 * dispatch packets); the call then waits for the stream.
 * Errors: EDB_ERR_INVALID, EDB_ERR_UNSUPPORTED (a batch inside a dataflow
 * launch), EDB_ERR_HIP. */
edb_status edb_split_phase_bytes(const edb_exec_t* e, int64_t* bytes);
edb_status edb_split_phase(edb_exec_t* e, const void* x, void* arena_h, void* arena_c, void* buf,
                           int64_t buf_bytes, void* stream, float* ms, int32_t n);

/* Roofline probes on the current device; each launches one kernel on
 * `stream`, waits for it and returns its duration in *ms (HIP events).
 * edb_probe_mfma: n_workgroups work-groups of 4 waves; each wave issues
 *   iters x 8 independent MFMAs on register operands, v_mfma_f32_16x16x4_f32
 *   (dtype EDB_F32, 2048 flops each) or v_mfma_f32_16x16x32_bf16 (EDB_BF16,
 *   16384 flops each).  out: device float[n_workgroups * 256] (the
 *   accumulators' sums, so the work is not dead).
 * edb_probe_copy: copies `bytes` (a multiple of 16) from src to dst with
 *   16-byte loads and stores, grid-stride over n_workgroups x 256 threads.
 * Errors: EDB_ERR_INVALID, EDB_ERR_HIP. */
edb_status edb_probe_mfma(int32_t dtype, int32_t n_workgroups, int32_t iters, float* out, void* stream,
                          float* ms);
edb_status edb_probe_copy(const void* src, void* dst, int64_t bytes, int32_t n_workgroups, void* stream,
                          float* ms);

void edb_exec_free(edb_exec_t* e);

#ifdef __cplusplus
}
#endif

#endif /* EDB_H */
