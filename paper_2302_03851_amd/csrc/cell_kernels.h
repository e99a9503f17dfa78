// Fused batch-cell kernels for gfx950 (MI355X).
//
// One launch executes one batch of the schedule (all ready nodes of one type,
// Algorithm 1 of ED-Batch): it gathers the operand rows of the batch, runs the
// cell's gate GEMM on the matrix cores, applies the gate nonlinearities and
// the cell-state update, and writes h and c into the planned arena slots.  The
// per-batch gather and scatter of Section 3.1 are therefore fused into the
// GEMM's prologue (operand rows staged through LDS, contiguous rows taking a
// base+row fast path) and epilogue (row-indexed stores).
//
// Work decomposition.  A work-group of WU*WK waves owns TM = 16*RT rows and
// TU = 16*WU hidden units of the batch, all G gates of those units.  Waves
// are split WU along units and WK along the reduction (split-K inside the
// work-group; partial sums are added in LDS in a fixed order, so the result
// does not depend on timing).  Each wave computes a 16*RT x 16 x G block with
// 16x16 MFMA tiles: v_mfma_f32_16x16x4_f32 (fp32) or v_mfma_f32_16x16x32_bf16
// (bf16 inputs, fp32 accumulation).  Small batches are latency bound, so the
// prologue issues every global load it can before waiting: operand rows in
// batches of 8 per thread, the epilogue's child cell states, and the first
// weight fragments; the GEMM loop keeps the weights of the next 2-4 k-groups
// in flight.
//
// Packed weights (gate-interleaved, zero padded; produced by edb_pack_weights):
//   main  [Hu/16 unit blocks][G gates][K/KG k-groups][64 lanes][16 bytes]
//   lane l of k-group kg holds, for unit u = ub*16 + l%16 of gate g, the KG/4
//   consecutive k values kg*KG + (l/16)*(KG/4) + i.  With KG = 16 (fp32) this
//   is 4 floats, one per MFMA of the k-group; with KG = 32 (bf16) 8 bf16
//   values, one MFMA operand.  One 16-byte load per lane per (gate, k-group).
//   bias  [G][Hu] fp32.  Ragged weights (child-sum U_f, lattice W_lc) use the
//   same layout with G = 1 and K = Hk.
// K layout of the A operand: [x (Ep)] [child 0 h (Hk)] [child 1 h (Hk)], each
// segment zero-padded to a multiple of KG; child-sum internal nodes use the
// child sum of h (Hk) as their only segment.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace edbk {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

enum { K_CHAIN = 0, K_NARY_LEAF = 1, K_NARY_INT = 2, K_GRID = 3, K_CS_LEAF = 4, K_CS_INT = 5,
       K_LAT_CHAR = 6, K_LAT_WORD = 7, K_GRU_LEAF = 8, K_GRU_INT = 9,
       // MV-RNN: a linear map (leaves), matrix columns, vectors (on rows [B a, A b])
       K_LINEAR = 10, K_MV_MAT = 11, K_MV_VEC = 12,
       // lattice GRU: an edge's GRU proposal, a position's mean over its edges
       K_LGRU_EDGE = 13, K_POOL_MEAN = 14,
       // the two GEMMs of a child-sum batch run on the large tile: the forget
       // gates over the batch's child rows, then the parents on their child sums
       K_CS_FORGET = 15, K_CS_PARENT = 16 };

enum { S_NONE = 0, S_CONTIG = 1, S_INDEXED = 2 };

// One operand list of a batch: entry r lives in row (kind == CONTIG ? base + r : idx[r]).
struct Seg {
    int kind;
    int base;
    const int* idx;
};

struct BatchArgs {
    int kind;         // cell kind (K_*)
    int m;            // rows in the batch
    int H, Hk, Hu;    // hidden size, its K-segment width (padded to KG), its unit padding (64)
    int E, Ep;        // input size and its padded K-segment width
    int K;            // total padded reduction length of the main GEMM
    Seg x;            // rows of the x matrix
    Seg fix[2];       // positional children (arena rows)
    Seg rag;          // ragged children (arena rows), entries rag_ptr[r] .. rag_ptr[r+1]
    const int* rag_ptr;
    Seg res;          // result rows
    const void* xmat;     // x (staged or caller's), row stride E
    const void* W;        // packed main weights
    const float* bias;    // packed main bias [G][Hu]
    const void* Wr;       // packed ragged weights
    const float* br;      // ragged bias [Hu]
    void* arena_h;        // [n_slots][H] of T
    float* arena_c;       // [n_slots][H]
    int n_slots;          // arena rows
    int n_xrows;          // rows of the x matrix xmat points to
    float* fc;            // child-sum batches on the large tile: sigma(f_k) * c_k per child, [children][H]
    const int* zrows;     // rows this launch clears in both arenas (the zero row and pads), or none
    int n_zero;
};


template <int KIND> struct Kind;
template <> struct Kind<K_CHAIN>    { static constexpr int G = 4, NFIX = 1; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_NARY_LEAF>{ static constexpr int G = 3, NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_NARY_INT> { static constexpr int G = 5, NFIX = 2; static constexpr bool X = false, RAG = false; };
template <> struct Kind<K_GRID>     { static constexpr int G = 5, NFIX = 2; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_CS_LEAF>  { static constexpr int G = 3, NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_CS_INT>   { static constexpr int G = 3, NFIX = 0; static constexpr bool X = false, RAG = true;  };
template <> struct Kind<K_LAT_CHAR> { static constexpr int G = 5, NFIX = 1; static constexpr bool X = true,  RAG = true;  };
template <> struct Kind<K_LAT_WORD> { static constexpr int G = 3, NFIX = 1; static constexpr bool X = true,  RAG = false; };
// TreeGRU: the node state is kept in the cell-state arena (children's states read like c rows)
template <> struct Kind<K_GRU_LEAF> { static constexpr int G = 2, NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_GRU_INT>  { static constexpr int G = 5, NFIX = 2; static constexpr bool X = false, RAG = false; };
// MV-RNN.  LINEAR: h = x W + b.  MV_MAT: rows = matrix columns j, operands =
// column j of the two children's matrices.  MV_VEC: x = the rows [B a, A b]
// that mv_matvec_kernel computes; h = tanh(x W + b).
template <> struct Kind<K_LINEAR>   { static constexpr int G = 1, NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_MV_MAT>   { static constexpr int G = 1, NFIX = 2; static constexpr bool X = false, RAG = false; };
template <> struct Kind<K_MV_VEC>   { static constexpr int G = 1, NFIX = 0; static constexpr bool X = true,  RAG = false; };
// Lattice GRU.  LGRU_EDGE: gates [z, r, n_x, n_h] over [x ; h_src] (n_x reads
// x only, n_h the source's h only).  POOL_MEAN: A = the sum of the ragged
// children's h (staged like a child-sum node), h = (A W + b) / children.
template <> struct Kind<K_LGRU_EDGE>{ static constexpr int G = 4, NFIX = 1; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_POOL_MEAN>{ static constexpr int G = 1, NFIX = 0; static constexpr bool X = false, RAG = false; };
// rows: the batch's children (x = their h rows); one gate
template <> struct Kind<K_CS_FORGET>{ static constexpr int G = 1, NFIX = 0; static constexpr bool X = true,  RAG = false; };
// rows: the parents (x = their child sums of h)
template <> struct Kind<K_CS_PARENT>{ static constexpr int G = 3, NFIX = 0; static constexpr bool X = true,  RAG = false; };

// Whether the cell update reads its positional children's cell states.
template <int KIND>
__host__ __device__ constexpr bool reads_child_c() { return KIND != K_MV_MAT; }
// Kinds whose A operand is the sum of the ragged children's h rows.
template <int KIND>
__host__ __device__ constexpr bool sums_children() { return KIND == K_CS_INT || KIND == K_POOL_MEAN; }

template <typename T> struct Elem;
template <> struct Elem<float>  { static constexpr int KG = 16; static constexpr int VEC = 4; };
template <> struct Elem<__bf16> { static constexpr int KG = 32; static constexpr int VEC = 8; };

// A-tile row padding in elements: 16 bytes, so that the 16 rows read by one
// MFMA operand load start in different LDS banks.
template <typename T> constexpr int a_pad() { return 16 / (int)sizeof(T); }
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int seg_row(const Seg& s, int r) {
    return s.kind == S_CONTIG ? s.base + r : s.idx[r];
}

// Gate nonlinearities from the hardware exponential (v_exp_f32) and
// reciprocal (v_rcp_f32), each about 1 ulp: the logistic function as
// 1 / (1 + e^-z), and tanh z = 1 - 2 / (1 + e^{2z}) (exact limits +-1 when the
// exponential overflows or vanishes).  Below |z| = 2^-9 tanh z = z to within
// z^3/3, under half an fp32 ulp of z, which also avoids the cancellation
// of the formula there.
__device__ __forceinline__ float sigm(float z) { return __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_f(float z) {
    const float t = fmaf(-2.0f, __builtin_amdgcn_rcpf(1.0f + __expf(2.0f * z)), 1.0f);
    return fabsf(z) < 0x1p-9f ? z : t;
}

// sigma(a) * tanh(b) from two exponentials and one reciprocal:
// sgn(b) (1 - q) / ((1 + p)(1 + q)) with p = e^-a and q = e^{-2|b|}.  q stays in
// (0, 1], and an overflowing p gives the exact limit 0; near b = 0 the error
// of 1 - q is absolute (about 1e-7), not relative.
__device__ __forceinline__ float sig_tanh(float a, float b) {
    const float p = __expf(-a);
    const float q = __expf(-2.0f * fabsf(b));
    const float den = fmaf(p, q, p + q) + 1.0f;
    return copysignf((1.0f - q) * __builtin_amdgcn_rcpf(den), b);
}

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(__bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ __bf16 from_f<__bf16>(float v) { return (__bf16)v; }

// The first batch's launch clears the arenas' zero row and pad rows when no
// staging launch runs before it.  That batch reads no arena row: nothing has
// run before it, so all of its child lists are absent, and it is used only for
// kinds without child lists, which never touch the zero row.  Every
// work-group takes a share, before any early exit.
template <typename T>
__device__ __forceinline__ void clear_zero_rows(const BatchArgs& a) {
    if (a.n_zero == 0) return;
    const int64_t n = (int64_t)a.n_zero * a.H;
    T* h = reinterpret_cast<T*>(a.arena_h);
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t o = (int64_t)a.zrows[i / a.H] * a.H + i % a.H;
        h[o] = from_f<T>(0.f);
        a.arena_c[o] = 0.f;
    }
}

// Gate nonlinearities and cell-state update of one (node, unit) element.
// z: the G gate pre-activations (bias included), cp: child cell states of the
// positional children, racc / rden: the ragged phase's sums (child-sum:
// sum_k f_k c_k; lattice: sum_k e^{l_k} c_w^k and sum_k e^{l_k}), nw: number
// of words ending at a lattice character.  Every multiply-add is an explicit
// fmaf (the library is compiled without floating-point contraction), so the
// update rounds identically in every kernel that uses it.
template <int KIND>
__device__ __forceinline__ void cell_update(const float* z, const float* cp, float racc, float rden, int nw,
                                            float& c, float& h) {
    if constexpr (KIND == K_CHAIN) {
        c = fmaf(sigm(z[1]), cp[0], sig_tanh(z[0], z[2]));
        h = sig_tanh(z[3], c);
    } else if constexpr (KIND == K_NARY_LEAF || KIND == K_CS_LEAF) {
        c = sig_tanh(z[0], z[2]);
        h = sig_tanh(z[1], c);
    } else if constexpr (KIND == K_NARY_INT || KIND == K_GRID) {
        c = fmaf(sigm(z[2]), cp[1], fmaf(sigm(z[1]), cp[0], sig_tanh(z[0], z[4])));
        h = sig_tanh(z[3], c);
    } else if constexpr (KIND == K_CS_INT) {
        c = sig_tanh(z[0], z[2]) + racc;
        h = sig_tanh(z[1], c);
    } else if constexpr (KIND == K_LAT_WORD) {
        c = fmaf(sigm(z[1]), cp[0], sig_tanh(z[0], z[2]));
        h = 0.f;
    } else if constexpr (KIND == K_GRU_LEAF) {   // gates [z, n]: (1 - sigma(z)) tanh(n)
        c = sig_tanh(-z[0], z[1]);
        h = c;
    } else if constexpr (KIND == K_GRU_INT) {    // gates [z, r_0, r_1, n_0, n_1]; cp: the children's states
        const float ht = tanh_f(fmaf(sigm(z[1]), z[3], sigm(z[2]) * z[4]));
        c = fmaf(sigm(z[0]), fmaf(0.5f, cp[0] + cp[1], -ht), ht);
        h = c;
    } else if constexpr (KIND == K_LINEAR || KIND == K_MV_MAT) {   // no nonlinearity; c mirrors h
        h = z[0];
        c = h;
    } else if constexpr (KIND == K_MV_VEC) {
        h = tanh_f(z[0]);
        c = h;
    } else if constexpr (KIND == K_LGRU_EDGE) {   // gates [z, r, n_x, n_h]; cp: the source position's state
        const float ht = tanh_f(fmaf(sigm(z[1]), z[3], z[2]));
        c = fmaf(sigm(z[0]), cp[0] - ht, ht);
        h = c;
    } else if constexpr (KIND == K_POOL_MEAN) {
        // nw: the position's edges; z[0] = (sum of their h) W without the
        // bias, which racc carries: mean(h) W + b (with no edge, b)
        c = (nw > 0 ? z[0] / (float)nw : 0.f) + racc;
        h = c;
    } else {  // K_LAT_CHAR: gates [i, f, o, u, lx]
        if (nw == 0) {
            c = fmaf(sigm(z[1]), cp[0], sig_tanh(z[0], z[3]));
        } else {
            const float e0 = __expf(sigm(z[0]));
            c = fmaf(e0, tanh_f(z[3]), racc) / (e0 + rden);
        }
        h = sig_tanh(z[2], c);
    }
}

// Row blocks per chunk of the ragged phase (child-sum children, lattice
// words): at least 4 (64 rows), so that the children of a tile's parents
// usually fit one chunk.
template <int KIND, int RT>
__host__ __device__ constexpr int rag_rt() {
    return Kind<KIND>::RAG ? (RT < 4 ? 4 : RT) : RT;
}

// Kinds whose first chunk of ragged rows (the lattice words ending at the
// tile's characters) is gathered together with the main A tile, into an LDS
// tile of its own, so that its loads overlap the main tile's and its GEMM
// follows the main GEMM without another round trip to memory.
template <int KIND>
__host__ __device__ constexpr bool early_rag() { return KIND == K_LAT_CHAR; }

// ---- LDS budget of one work-group (bytes); Hk: the ragged rows' width ----
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_a_bytes(int K, int Hk) {
    if (early_rag<KIND>())   // main tile, then the ragged tile [16*rag_rt rows][Hk + pad]
        return (16 * RT * (K + a_pad<T>()) + 16 * rag_rt<KIND, RT>() * (Hk + a_pad<T>())) * (int)sizeof(T);
    // other ragged kinds reuse A for the chunk's child rows (Hk <= K columns)
    return 16 * rag_rt<KIND, RT>() * (K + a_pad<T>()) * (int)sizeof(T);
}
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_z_bytes() {
    return WK * 16 * RT * Kind<KIND>::G * 16 * WU * 4;
}
// Zr (the chunk's per-child GEMM partials) and Crag (its cell states)
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_zr_bytes() {
    return Kind<KIND>::RAG ? (WK + 1) * 16 * rag_rt<KIND, RT>() * 16 * WU * 4 : 0;
}
// Offset of Z: after A for kinds with a ragged phase (A is reused for child
// rows while Z must persist), else Z aliases A (written after the GEMM).
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_z_off(int K, int Hk) {
    return Kind<KIND>::RAG ? lds_a_bytes<KIND, T, RT, WU, WK>(K, Hk) : 0;
}
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_rowc_off(int K, int Hk) {
    return Kind<KIND>::RAG
               ? lds_a_bytes<KIND, T, RT, WU, WK>(K, Hk) + lds_z_bytes<KIND, T, RT, WU, WK>() +
                     lds_zr_bytes<KIND, T, RT, WU, WK>()
               : (lds_a_bytes<KIND, T, RT, WU, WK>(K, Hk) > lds_z_bytes<KIND, T, RT, WU, WK>()
                      ? lds_a_bytes<KIND, T, RT, WU, WK>(K, Hk)
                      : lds_z_bytes<KIND, T, RT, WU, WK>());
}
template <int KIND, typename T, int RT, int WU, int WK>
__host__ __device__ constexpr int lds_bytes(int K, int Hk) {
    return lds_rowc_off<KIND, T, RT, WU, WK>(K, Hk);
}

// Raw buffer resource over `bytes` bytes at p (gfx9 resource word 3).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// 16-byte buffer load at byte offset off; zero past the end of the buffer.
__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0));
}
// 4-byte buffer load at byte offset off; zero past the end of the buffer.
__device__ __forceinline__ uint32_t bload32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
}
// seg_row without a branch: an indexed list is read through a buffer of the
// batch's m entries (zero past them), a list of another kind reads nothing.
// Several of these issue their loads back to back and are waited for once.
__device__ __forceinline__ int seg_row_nb(const Seg& s, int r, int m) {
    const __amdgpu_buffer_rsrc_t ri = make_rsrc(s.idx, s.kind == S_INDEXED ? (uint32_t)m * 4u : 0u);
    const int v = (int)bload32(ri, (uint32_t)r * 4u);
    return s.kind == S_CONTIG ? s.base + r : v;
}

// One K segment of the A tile: tile row r reads source row
// seg_row(seg, row0 + r) (zeros when the list is absent), `nreal` 16-byte
// chunks of data (row stride `width` elements), zero up to `nv` chunks.
// Contiguous lists need no index load at all.
template <typename T>
struct ASeg {
    const T* src;
    Seg seg;
    int row0;
    int col;        // first chunk of the segment in the tile row
    int nv;         // chunks of the (padded) segment
    int nreal;      // chunks holding data
    int width;      // source row stride (elements)
    int len;        // entries of the row list
};

// Stage the first nrows rows of the A tile [TM rows][nseg segments] (rows past
// them are left as they are: each output row depends on its own A row only,
// and the epilogue skips them), one segment at a time, in rounds of up to SR
// items per thread (4: the staged values share the registers with the weight
// ring already in flight): the round's row indices are loaded back to back
// without branches (seg_row_nb), then its 16-byte pieces, then stored to LDS.
// A piece past the data (the zero padding of K) or of an absent list reads 16
// bytes of `zero` (the arena's zero row) instead of branching around its
// load, so the round's loads issue back to back and are waited for once.
template <typename T, int TM, int NT, int NSEG, int SR = 4>
__device__ __forceinline__ void stage_tile(T* A, int AS, const ASeg<T> (&sg)[NSEG], int nrows, const T* zero,
                                           int tid) {
    constexpr int V = Elem<T>::VEC;
#pragma unroll
    for (int s = 0; s < NSEG; ++s) {
        const ASeg<T>& q = sg[s];
        const int total = nrows * q.nv;
        for (int base = 0; base < total; base += NT * SR) {
            int row[SR];
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = min(base + i * NT + tid, total - 1);
                row[i] = seg_row_nb(q.seg, q.row0 + it / q.nv, q.len);
            }
            u32x4 val[SR];   // a vector type: struct copies of uint4 kept the array in scratch
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = base + i * NT + tid, r = it / q.nv, c = it - r * q.nv;
                const bool ok = it < total && c < q.nreal && q.seg.kind != S_NONE;
                val[i] = *reinterpret_cast<const u32x4*>(ok ? q.src + (size_t)row[i] * q.width + c * V : zero);
            }
            // keeps the loads together (the compiler would sink each into its store's branch)
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = base + i * NT + tid, r = it / q.nv, c = it - r * q.nv;
                if (it < total) *reinterpret_cast<u32x4*>(A + r * AS + (q.col + c) * V) = val[i];
            }
        }
    }
}

// Segment-parallel staging of the A tile for kinds with early loads: round
// `base` takes up to SR items of every segment per thread, all their row
// indices first (idx, descriptor data only), then all their 16-byte pieces
// (vals), then the LDS stores (store), so that a tile whose segments fit one
// round costs one index and one data round trip however many segments it
// has, and the indices can be issued before the wait for the producers.
template <typename T, int NSEG, int SR>
struct StageRound {
    int row[NSEG][SR];
    u32x4 val[NSEG][SR];

    template <int NT>
    __device__ __forceinline__ void idx(const ASeg<T> (&sg)[NSEG], int nrows, int base, int tid) {
#pragma unroll
        for (int s = 0; s < NSEG; ++s) {
            const int total = nrows * sg[s].nv;
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = min(base + i * NT + tid, total - 1);
                row[s][i] = seg_row_nb(sg[s].seg, sg[s].row0 + it / sg[s].nv, sg[s].len);
            }
        }
    }
    template <int NT>
    __device__ __forceinline__ void vals(const ASeg<T> (&sg)[NSEG], int nrows, int base, const T* zero, int tid) {
        constexpr int V = Elem<T>::VEC;
#pragma unroll
        for (int s = 0; s < NSEG; ++s) {
            const ASeg<T>& q = sg[s];
            const int total = nrows * q.nv;
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = base + i * NT + tid, r = it / q.nv, c = it - r * q.nv;
                const bool ok = it < total && c < q.nreal && q.seg.kind != S_NONE;
                val[s][i] = *reinterpret_cast<const u32x4*>(ok ? q.src + (size_t)row[s][i] * q.width + c * V : zero);
            }
        }
    }
    template <int NT>
    __device__ __forceinline__ void store(T* A, int AS, const ASeg<T> (&sg)[NSEG], int nrows, int base, int tid) const {
        constexpr int V = Elem<T>::VEC;
#pragma unroll
        for (int s = 0; s < NSEG; ++s) {
            const ASeg<T>& q = sg[s];
            const int total = nrows * q.nv;
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = base + i * NT + tid, r = it / q.nv, c = it - r * q.nv;
                if (it < total) *reinterpret_cast<u32x4*>(A + r * AS + (q.col + c) * V) = val[s][i];
            }
        }
    }
};

// Child sum of h rows for child-sum internal nodes and pooling nodes:
// A[r][k] = the sum of the row's ragged children's h[k], added in child order
// in fp32 and rounded to T once.  Items (row, 16-byte piece) are taken SR per
// thread at a time: bounds() loads their rows' child ranges (descriptor data,
// issued with the tile's other indices, before the wait for the producers);
// gather() takes the children CB at a time for all SR items, their row
// indices back to back, then their pieces (a slot past an item's last child
// reads the zero row and is not added), then stores the sums.  A round costs
// one index and one data round trip per CB children of its largest parent.
template <typename T, int NT, int SR, int CB>
struct ChildSum {
    int e0[SR], e1[SR];

    __device__ __forceinline__ void bounds(const BatchArgs& a, int row0, int nrows, int base, int tid) {
        const int nv = a.Hk / Elem<T>::VEC, nreal = a.H / Elem<T>::VEC, total = nrows * nv;
#pragma unroll
        for (int i = 0; i < SR; ++i) {
            const int it = base + i * NT + tid, itc = min(it, total - 1);
            const int r = itc / nv, c = itc - r * nv;
            const int p0 = a.rag_ptr[row0 + r], p1 = a.rag_ptr[row0 + r + 1];
            e0[i] = p0;
            e1[i] = it < total && c < nreal ? p1 : p0;   // zero padding and past the tile: no children
        }
    }
    __device__ __forceinline__ void gather(T* A, int AS, const BatchArgs& a, int nrows, int base, int tid) const {
        constexpr int V = Elem<T>::VEC;
        const T* h = reinterpret_cast<const T*>(a.arena_h);
        const int nv = a.Hk / V, total = nrows * nv;
        float acc[SR][V];
        int n = 0;
#pragma unroll
        for (int i = 0; i < SR; ++i) {
            n = max(n, e1[i] - e0[i]);
#pragma unroll
            for (int k = 0; k < V; ++k) acc[i][k] = 0.f;
        }
        for (int j = 0; j < n; j += CB) {
            int row[SR][CB];
#pragma unroll
            for (int i = 0; i < SR; ++i)
#pragma unroll
                for (int q = 0; q < CB; ++q) row[i][q] = seg_row_nb(a.rag, min(e0[i] + j + q, e1[i] - 1), e1[i]);
            u32x4 raw[SR][CB];
#pragma unroll
            for (int i = 0; i < SR; ++i) {
                const int it = min(base + i * NT + tid, total - 1), c = it - (it / nv) * nv;
#pragma unroll
                for (int q = 0; q < CB; ++q)
                    raw[i][q] = *reinterpret_cast<const u32x4*>(
                        e0[i] + j + q < e1[i] ? h + (size_t)row[i][q] * a.H + c * V : h);
            }
#pragma unroll
            for (int i = 0; i < SR; ++i)
#pragma unroll
                for (int q = 0; q < CB; ++q) {
                    const T* pv = reinterpret_cast<const T*>(&raw[i][q]);
                    if (e0[i] + j + q < e1[i])
#pragma unroll
                        for (int k = 0; k < V; ++k) acc[i][k] += to_f(pv[k]);
                }
        }
#pragma unroll
        for (int i = 0; i < SR; ++i) {
            const int it = base + i * NT + tid, r = it / nv, c = it - r * nv;
            if (it >= total) continue;
            uint4 out;
            T* po = reinterpret_cast<T*>(&out);
#pragma unroll
            for (int k = 0; k < V; ++k) po[k] = from_f<T>(acc[i][k]);
            *reinterpret_cast<uint4*>(A + r * AS + c * V) = out;
        }
    }
};

// Lattice words' cell states c_w (fp32 arena rows of the ragged list entries
// [cb, cb + cn)) converted to T into the ragged tile R (stride RS), pieces
// [base0, cn * Hk / VEC) of V elements, two per thread a round: indices,
// then values (past H: the zero row), then the converted stores.
template <typename T, int NT>
__device__ __forceinline__ void stage_word_rows(T* R, int RS, const BatchArgs& a, int cb, int cn, int base0, int tid) {
    constexpr int V = Elem<T>::VEC;
    const int nv = a.Hk / V, nreal = a.H / V, total = cn * nv;   // rows past cn are not read back
    for (int base = base0; base < total; base += 2 * NT) {
        int wr[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int it = min(base + q * NT + tid, total - 1);
            wr[q] = seg_row_nb(a.rag, cb + min(it / nv, cn - 1), cb + cn);
        }
        float4 f4[2][V / 4];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int it = base + q * NT + tid, r = it / nv, c = it - r * nv;
            const bool ok = it < total && c < nreal;
            const float4* src = reinterpret_cast<const float4*>(ok ? a.arena_c + (size_t)wr[q] * a.H + c * V : a.arena_c);
#pragma unroll
            for (int k = 0; k < V / 4; ++k) f4[q][k] = src[k];
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int it = base + q * NT + tid, r = it / nv, c = it - r * nv;
            if (it >= total) continue;
            uint4 out;
            T* po = reinterpret_cast<T*>(&out);
            const float* pf = reinterpret_cast<const float*>(&f4[q][0]);
#pragma unroll
            for (int i = 0; i < V; ++i) po[i] = from_f<T>(pf[i]);
            *reinterpret_cast<uint4*>(R + r * RS + c * V) = out;
        }
    }
}

// MFMA on one (gate, row-block) accumulator for one k-group.
template <typename T, int G, int RT>
__device__ __forceinline__ void kgroup_mma(v4f (&acc)[G][RT], const uint4 (&av)[RT], const uint4 (&bv)[G]) {
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const float a_ = __uint_as_float((&av[rt].x)[j]);
                    const float b_ = __uint_as_float((&bv[g].x)[j]);
                    acc[g][rt] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_, b_, acc[g][rt], 0, 0, 0);
                }
    } else {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                v8bf a_ = __builtin_bit_cast(v8bf, av[rt]);
                v8bf b_ = __builtin_bit_cast(v8bf, bv[g]);
                acc[g][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_, b_, acc[g][rt], 0, 0, 0);
            }
    }
}

// Weight fragments of k-group kg for all gates (B points at this lane's
// (ub, gate 0, k-group 0) chunk).
template <int G>
__device__ __forceinline__ void load_b(uint4 (&bv)[G], const uint4* B, int nkg, int kg) {
#pragma unroll
    for (int g = 0; g < G; ++g) bv[g] = B[((size_t)g * nkg + kg) * 64];
}

// Weight prefetch ring: PD k-groups of fragments in flight.
template <int G> constexpr int ring_depth() { return G >= 5 ? 3 : 4; }
template <int G, int PD>
struct BRing {
    uint4 b[PD][G];
};

template <int G, int PD>
__device__ __forceinline__ void ring_prologue(BRing<G, PD>& r, const uint4* B, int nkg, int kg0, int kg1) {
    if (kg0 >= kg1) return;
#pragma unroll
    for (int s = 0; s < PD; ++s) load_b<G>(r.b[s], B, nkg, min(kg0 + s, kg1 - 1));
}

// A fragments of k-group k for all row blocks of the wave.
template <typename T, int RT>
__device__ __forceinline__ void load_a(uint4 (&av)[RT], const T* A, int AS, int k, int lane) {
    constexpr int KG = Elem<T>::KG;
    const int arow = lane & 15, aq = lane >> 4;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
        av[rt] = *reinterpret_cast<const uint4*>(A + (rt * 16 + arow) * AS + k * KG + aq * (KG / 4));
}

// GEMM of one wave over k-groups [kg0, kg1): acc[g][rt] += A[rt*16 .. +16] * W[ub][g].
// The ring holds k-groups kg0 .. kg0+PD-1 on entry (ring_prologue; indices
// past the end repeat the last k-group).  In the steady state every slot is
// refilled, unconditionally, with the k-group PD steps ahead (clamped to the
// last one), so the compiler can wait for exactly the load a slot needs; the
// remaining k-groups drain the ring without loads.
template <typename T, int G, int RT, int PD>
__device__ __forceinline__ void wave_gemm(v4f (&acc)[G][RT], const T* A, int AS, const uint4* B, int nkg,
                                          int kg0, int kg1, int lane, BRing<G, PD>& ring) {
    int kg = kg0;
    for (; kg + PD < kg1; kg += PD) {
        uint4 av[PD][RT];
#pragma unroll
        for (int s = 0; s < PD; ++s) load_a<T, RT>(av[s], A, AS, kg + s, lane);
#pragma unroll
        for (int s = 0; s < PD; ++s) {
            kgroup_mma<T, G, RT>(acc, av[s], ring.b[s]);
            load_b<G>(ring.b[s], B, nkg, min(kg + s + PD, kg1 - 1));
        }
    }
    uint4 av[PD][RT];
#pragma unroll
    for (int s = 0; s < PD; ++s)
        if (kg + s < kg1) load_a<T, RT>(av[s], A, AS, kg + s, lane);
#pragma unroll
    for (int s = 0; s < PD; ++s)
        if (kg + s < kg1) kgroup_mma<T, G, RT>(acc, av[s], ring.b[s]);
}

// No inter-tile synchronisation (one launch per batch: kernel boundaries order
// producers before consumers).
struct NoSync {
    __device__ __forceinline__ void wait() const {}
    __device__ __forceinline__ void signal() const {}
};

// One tile: rows [16*RT*rtile, +16*RT) x units [16*WU*ut, +16*WU) of a batch,
// all gates.  sync.wait() runs after the weight and descriptor loads and
// before the first read of a producer's output; sync.signal() after the
// tile's h and c stores.
template <int KIND, typename T, int RT, int WU, int WK, typename Sync>
__device__ __forceinline__ void cell_tile(const BatchArgs& a, int rtile, int ut, char* smem, const Sync& sync) {
    using KT = Kind<KIND>;
    constexpr int G = KT::G;
    constexpr int NT = 64 * WU * WK;
    constexpr int TM = 16 * RT, TU = 16 * WU;
    constexpr int KG = Elem<T>::KG;
    constexpr int AS_PAD = a_pad<T>();
    constexpr int NITEM = TM * TU;
    constexpr int NI = (NITEM + NT - 1) / NT;     // epilogue items per thread
    constexpr int NFX = KT::NFIX;

    const int AS = a.K + AS_PAD;                           // A row stride (elements)
    constexpr int TMR = 16 * rag_rt<KIND, RT>();           // rows per chunk of the ragged phase
    constexpr bool ER = early_rag<KIND>();
    constexpr bool CSUM = sums_children<KIND>();
    // kinds that load their biases and child ranges with the row indices
    // (their work-groups hold one per CU, with registers to spare)
    constexpr bool EARLY = KT::RAG || CSUM;
    T* A = reinterpret_cast<T*>(smem);
    T* Ar = ER ? A + TM * AS : A;                          // the ragged chunk's rows
    const int RS = a.Hk + AS_PAD;                          // their row stride
    float* Z = reinterpret_cast<float*>(smem + lds_z_off<KIND, T, RT, WU, WK>(a.K, a.Hk));
    float* Zr = Z + WK * TM * G * TU;
    float* Crag = Zr + WK * TMR * TU;
    constexpr int PD = WK >= 16 ? 2 : ring_depth<G>();   // 1024-thread groups have 128 VGPRs
    constexpr int V = Elem<T>::VEC;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int row0 = rtile * TM, u0 = ut * TU;
    const int nrows = min(TM, a.m - row0);
    const int wu = wave % WU, wk = wave / WU;
    const int nkg = a.K / KG;
    const int ub = u0 / 16 + wu;
    const uint4* Bmain = reinterpret_cast<const uint4*>(a.W) + ((size_t)ub * G * nkg) * 64 + lane;
    const int kg0 = (nkg * wk) / WK, kg1 = (nkg * (wk + 1)) / WK;

    // first weight fragments: independent of everything, issued first
    BRing<G, PD> ring;
    ring_prologue<G, PD>(ring, Bmain, nkg, kg0, kg1);

    // the ragged phase's weights (W_lc for the early chunk: issued now) and
    // the tile's child range [cbeg, cend) (uniform)
    const int nkgr = KT::RAG ? a.Hk / KG : 0;
    const uint4* Brag = nullptr;
    if constexpr (KT::RAG) Brag = reinterpret_cast<const uint4*>(a.Wr) + ((size_t)ub * nkgr) * 64 + lane;
    const int rk0 = (nkgr * wk) / WK, rk1 = (nkgr * (wk + 1)) / WK;
    BRing<1, 4> rring;
    int cbeg = 0, cend = 0;
    if constexpr (KT::RAG) {
        cbeg = a.rag_ptr[row0];
        cend = a.rag_ptr[row0 + nrows];
    }
    if constexpr (ER) ring_prologue<1, 4>(rring, Brag, nkgr, rk0, rk1);

    // ---- 1. early loads: the epilogue's result rows and child cell states ----
    // (row indices of contiguous lists are arithmetic; indexed lists cost one
    // load, issued here in parallel with the operand and weight loads)
    // (branch-free: the lookups of a thread issue back to back; a masked
    // cell state reads the zero row instead of branching around its load)
    int rres[NI], crow[NI][NFX > 0 ? NFX : 1];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int rr = row0 + min(tid + NT * q, NITEM - 1) / TU;
        rres[q] = seg_row_nb(a.res, rr, a.m);
#pragma unroll
        for (int p = 0; p < NFX; ++p) crow[q][p] = seg_row_nb(a.fix[p], rr, a.m);
    }
    // biases (the packed ones are padded to Hu) and each item's child range
    float bz[NI][G], brj[NI];
    int pe0[NI], pe1[NI];
    if constexpr (EARLY) {
#pragma unroll
        for (int q = 0; q < NI; ++q) {
            const int it = tid + NT * q, itc = it < NITEM ? it : 0;
            const int r = itc / TU, u = itc % TU;
#pragma unroll
            for (int g = 0; g < G; ++g) bz[q][g] = a.bias[g * a.Hu + u0 + u];
            if constexpr (KT::RAG) brj[q] = a.br[u0 + u];
            const int rr = row0 + min(r, nrows - 1);
            const int p0 = a.rag_ptr[rr], p1 = a.rag_ptr[rr + 1];
            const bool ok = it < NITEM && r < nrows;
            pe0[q] = ok ? p0 : 0;
            pe1[q] = ok ? p1 : 0;
        }
    }
    // the main A tile's sources: [x | child h ...] (kinds that do not sum children)
    constexpr int NSEG = (KT::X ? 1 : 0) + NFX;
    constexpr int NS1 = NSEG > 0 ? NSEG : 1;   // the kinds that sum children have no segments
    ASeg<T> sg[NS1];
    if constexpr (!CSUM) {
        int s = 0, col = 0;
        if constexpr (KT::X) {
            sg[s++] = ASeg<T>{reinterpret_cast<const T*>(a.xmat), a.x, row0, 0, a.Ep / V, a.E / V, a.E, a.m};
            col += a.Ep / V;
        }
#pragma unroll
        for (int p = 0; p < NFX; ++p) {
            // an absent operand list reads the zero row 0
            sg[s++] = ASeg<T>{reinterpret_cast<const T*>(a.arena_h), a.fix[p], row0, col, a.Hk / V, a.H / V, a.H, a.m};
            col += a.Hk / V;
        }
    }
    constexpr int SR = 4;
    ChildSum<T, NT, SR, KT::RAG ? 4 : 2> csum;   // pooling nodes: 168 registers a lane
    if constexpr (CSUM) csum.bounds(a, row0, nrows, 0, tid);
    StageRound<T, NS1, SR> st;
    if constexpr (ER) st.template idx<NT>(sg, nrows, 0, tid);
    // the early ragged chunk's row indices: its cell states for this tile's
    // units (Crag) and the first NWQ pieces per thread of its rows (Ar)
    constexpr int NCI = (TMR * TU + NT - 1) / NT;
    constexpr int NWQ = 4;
    const int cn0 = min(TMR, cend - cbeg);
    const int nvr = a.Hk / V, total0 = cn0 * nvr;
    int crw[NCI], wr[NWQ];
    if constexpr (ER) {
#pragma unroll
        for (int q = 0; q < NCI; ++q) {
            const int it = min(tid + NT * q, TMR * TU - 1);
            crw[q] = seg_row_nb(a.rag, cbeg + min(it / TU, max(cn0 - 1, 0)), cbeg + cn0);
        }
#pragma unroll
        for (int q = 0; q < NWQ; ++q) {
            const int it = min(q * NT + tid, max(total0 - 1, 0));
            wr[q] = seg_row_nb(a.rag, cbeg + min(it / nvr, max(cn0 - 1, 0)), cbeg + cn0);
        }
    }
    sync.wait();   // producers of this tile's operand rows have finished

    // ---- 2. stage the A tile: [x | child h ...] or [child sum of h] ----
    float cv[NCI];
    float4 f4[NWQ][V / 4];
    const T* zero = reinterpret_cast<const T*>(a.arena_h);
    if constexpr (CSUM) {
        csum.gather(A, AS, a, nrows, 0, tid);
        for (int base = NT * SR; base < nrows * nvr; base += NT * SR) {
            csum.bounds(a, row0, nrows, base, tid);
            csum.gather(A, AS, a, nrows, base, tid);
        }
    } else if constexpr (ER) {
        st.template vals<NT>(sg, nrows, 0, zero, tid);
        // the early chunk's values (masked: the zero row), behind the tile's
#pragma unroll
        for (int q = 0; q < NCI; ++q) {
            const int it = tid + NT * q, j = u0 + it % TU;
            const bool ok = it < cn0 * TU && j < a.H;
            cv[q] = *(ok ? a.arena_c + (size_t)crw[q] * a.H + j : a.arena_c);
        }
#pragma unroll
        for (int q = 0; q < NWQ; ++q) {
            const int it = q * NT + tid, r = it / nvr, c = it - r * nvr;
            const bool ok = it < total0 && c < a.H / V;
            const float4* src = reinterpret_cast<const float4*>(ok ? a.arena_c + (size_t)wr[q] * a.H + c * V : a.arena_c);
#pragma unroll
            for (int k = 0; k < V / 4; ++k) f4[q][k] = src[k];
        }
        __builtin_amdgcn_sched_barrier(0);
        st.template store<NT>(A, AS, sg, nrows, 0, tid);
        int nmax = 0;
#pragma unroll
        for (int s = 0; s < NSEG; ++s) nmax = max(nmax, nrows * sg[s].nv);
        for (int base = NT * SR; base < nmax; base += NT * SR) {
            st.template idx<NT>(sg, nrows, base, tid);
            st.template vals<NT>(sg, nrows, base, zero, tid);
            __builtin_amdgcn_sched_barrier(0);
            st.template store<NT>(A, AS, sg, nrows, base, tid);
        }
    } else {
        stage_tile<T, TM, NT, NSEG>(A, AS, sg, nrows, zero, tid);
    }
    // the children's cell states: only the epilogue reads them, so they are
    // loaded behind the operand rows
    float cpre[NI][NFX > 0 ? NFX : 1];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + NT * q, r = it / TU, j = u0 + it % TU;
        const bool ok = it < NITEM && r < nrows && j < a.H;
#pragma unroll
        for (int p = 0; p < (NFX > 0 ? NFX : 1); ++p) {
            const bool use = NFX > p && reads_child_c<KIND>() && ok && a.fix[p].kind != S_NONE;
            cpre[q][p] = *(use ? a.arena_c + (size_t)crow[q][p] * a.H + j : a.arena_c);
        }
    }
    __syncthreads();

    // ---- 3. gate GEMM: wave (wu, wk) -> unit block ub, k-groups [kg0, kg1) ----
    {
        v4f acc[G][RT];
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[g][rt] = v4f{0.f, 0.f, 0.f, 0.f};
        if (kg0 < kg1) wave_gemm<T, G, RT, PD>(acc, A, AS, Bmain, nkg, kg0, kg1, lane, ring);
        if constexpr (!KT::RAG) __syncthreads();   // Z aliases A: all waves done reading A
        // partial sums -> Z[wk][row][g][unit]
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int r = rt * 16 + (lane >> 4) * 4 + i;
                    const int u = wu * 16 + (lane & 15);
                    Z[((wk * TM + r) * G + g) * TU + u] = acc[g][rt][i];
                }
    }

    // the ragged phase's per-child GEMM of rows [cb, cb + cn) staged in Ar:
    // partials -> Zr[wk][row][unit]
    // (only the row blocks holding rows: a chunk of a few words takes one)
    auto rag_gemm = [&](int cn) {
        constexpr int RTR = TMR / 16;
        v4f acc[1][RTR];
#pragma unroll
        for (int rt = 0; rt < RTR; ++rt) acc[0][rt] = v4f{0.f, 0.f, 0.f, 0.f};
        if (rk0 < rk1 && cn > 0) {
            if (RTR > 1 && cn <= 16) {
                v4f a1[1][1] = {{v4f{0.f, 0.f, 0.f, 0.f}}};
                wave_gemm<T, 1, 1, 4>(a1, Ar, RS, Brag, nkgr, rk0, rk1, lane, rring);
                acc[0][0] = a1[0][0];
            } else if (RTR > 2 && cn <= 32) {
                v4f a2[1][2] = {{v4f{0.f, 0.f, 0.f, 0.f}, v4f{0.f, 0.f, 0.f, 0.f}}};
                wave_gemm<T, 1, 2, 4>(a2, Ar, RS, Brag, nkgr, rk0, rk1, lane, rring);
                acc[0][0] = a2[0][0];
                acc[0][1] = a2[0][1];
            } else {
                wave_gemm<T, 1, RTR, 4>(acc, Ar, RS, Brag, nkgr, rk0, rk1, lane, rring);
            }
        }
#pragma unroll
        for (int rt = 0; rt < RTR; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rt * 16 + (lane >> 4) * 4 + i;
                const int u = wu * 16 + (lane & 15);
                Zr[(wk * TMR + r) * TU + u] = acc[0][rt][i];
            }
    };
    if constexpr (ER) {
        // the early chunk: cell states to Crag, rows converted to T into Ar
        // (pieces beyond the early ones loaded now), then its GEMM
#pragma unroll
        for (int q = 0; q < NCI; ++q)   // rows past cn0 are never read
            if (tid + NT * q < cn0 * TU) Crag[tid + NT * q] = cv[q];
#pragma unroll
        for (int q = 0; q < NWQ; ++q) {
            const int it = q * NT + tid, r = it / nvr, c = it - r * nvr;
            if (it >= total0) continue;
            uint4 out;
            T* po = reinterpret_cast<T*>(&out);
            const float* pf = reinterpret_cast<const float*>(&f4[q][0]);
#pragma unroll
            for (int i = 0; i < V; ++i) po[i] = from_f<T>(pf[i]);
            *reinterpret_cast<uint4*>(Ar + r * RS + c * V) = out;
        }
        stage_word_rows<T, NT>(Ar, RS, a, cbeg, cn0, NWQ * NT, tid);
        __syncthreads();
        rag_gemm(cn0);
    }
    __syncthreads();

    // ---- 4. per-item gate pre-activations (fixed-order sum over the K split) ----
    float zsum[NI][G];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + NT * q;
        const int r = (it < NITEM ? it : 0) / TU, u = (it < NITEM ? it : 0) % TU;
        const int j = u0 + u;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < WK; ++w) s += Z[((w * TM + r) * G + g) * TU + u];
            // a pooling node adds its bias after the mean (in the epilogue)
            const float b = EARLY ? bz[q][g] : a.bias[g * a.Hu + j];
            zsum[q][g] = KIND == K_POOL_MEAN ? s : s + b;
        }
    }

    // ---- 5. ragged phase: per-child GEMM (child-sum U_f, lattice W_lc) ----
    float racc[NI], rden[NI];
#pragma unroll
    for (int q = 0; q < NI; ++q) { racc[q] = 0.f; rden[q] = 0.f; }
    if constexpr (KIND == K_POOL_MEAN) {
#pragma unroll
        for (int q = 0; q < NI; ++q) racc[q] = bz[q][0];
    }
    if constexpr (KT::RAG) {
        // each item's children (words) among rows [cb, cb + cn): the per-child
        // sums from Zr, their cell states from Crag
        auto accumulate = [&](int cb, int cn) {
#pragma unroll
            for (int q = 0; q < NI; ++q) {
                const int it = tid + NT * q, u = it % TU;
                const int j = u0 + u;
                if (j >= a.H) continue;
                const int e0 = max(pe0[q], cb), e1 = min(pe1[q], cb + cn);
                for (int e = e0; e < e1; ++e) {
                    float s = brj[q];
#pragma unroll
                    for (int w = 0; w < WK; ++w) s += Zr[(w * TMR + (e - cb)) * TU + u];
                    const float cw = Crag[(e - cb) * TU + u];
                    if constexpr (KIND == K_CS_INT) {
                        racc[q] += sigm(s) * cw;   // f_k * c_k, rounded, then added in child order
                    } else {
                        const float l = sigm(zsum[q][4] + s);  // link gate of word k
                        const float ek = __expf(l);
                        racc[q] = fmaf(ek, cw, racc[q]);
                        rden[q] += ek;
                    }
                }
            }
        };
        if constexpr (ER) accumulate(cbeg, cn0);
        // the remaining chunks of TMR rows: their h rows (child-sum) or cell
        // states (lattice) staged to Ar, their cell states for this tile's
        // units to Crag, the per-child GEMM to Zr
        for (int cb = ER ? cbeg + TMR : cbeg; cb < cend; cb += TMR) {
            const int cn = min(TMR, cend - cb);
            __syncthreads();   // previous chunk's readers of Ar / Zr / Crag are done
            ring_prologue<1, 4>(rring, Brag, nkgr, rk0, rk1);
            {   // the chunk's cell states: indices, then values (masked: the zero row), then stores
                int crx[NCI];
                float cvx[NCI];
#pragma unroll
                for (int q = 0; q < NCI; ++q) {
                    const int it = min(tid + NT * q, TMR * TU - 1);
                    crx[q] = seg_row_nb(a.rag, cb + min(it / TU, cn - 1), cb + cn);
                }
#pragma unroll
                for (int q = 0; q < NCI; ++q) {
                    const int it = tid + NT * q, j = u0 + it % TU;
                    const bool ok = it < cn * TU && j < a.H;
                    cvx[q] = *(ok ? a.arena_c + (size_t)crx[q] * a.H + j : a.arena_c);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = 0; q < NCI; ++q)   // rows past cn are never read
                    if (tid + NT * q < cn * TU) Crag[tid + NT * q] = cvx[q];
            }
            if constexpr (KIND == K_CS_INT) {
                ASeg<T> sr[1] = {ASeg<T>{reinterpret_cast<const T*>(a.arena_h), a.rag, cb, 0, a.Hk / V, a.H / V, a.H,
                                         cb + cn}};
                stage_tile<T, TMR, NT, 1>(Ar, RS, sr, cn, zero, tid);
            } else {
                stage_word_rows<T, NT>(Ar, RS, a, cb, cn, 0, tid);
            }
            __syncthreads();
            rag_gemm(cn);
            __syncthreads();
            accumulate(cb, cn);
        }
    }

    // ---- 6. gate epilogue and scatter of h, c ----
    T* Hout = reinterpret_cast<T*>(a.arena_h);
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + NT * q, r = it / TU, u = it % TU;
        const int j = u0 + u;
        if (it >= NITEM || r >= nrows || j >= a.H) continue;
        float c, h;
        // words ending at a lattice character, edges of a pooled position
        cell_update<KIND>(zsum[q], cpre[q], racc[q], rden[q],
                          KIND == K_LAT_CHAR || KIND == K_POOL_MEAN ? pe1[q] - pe0[q] : 0, c, h);
        const size_t o = (size_t)rres[q] * a.H + j;
        a.arena_c[o] = c;
        Hout[o] = from_f<T>(h);
    }
    sync.signal();
}

// One launch per batch: work-group -> (row tile, unit tile).  Work-groups of
// 4 waves without a ragged phase (and not 32 rows x 64 units, which would
// spill) ask for at least 3 waves per SIMD (at most 168 registers a lane): 3
// such work-groups per CU, so batches of up to 768 tiles run in one round
// (unbounded, the compiler used up to 220 registers, 2 work-groups per CU).
template <int KIND, typename T, int RT, int WU, int WK>
__global__ __launch_bounds__(64 * WU * WK, WU * WK == 4 && RT * WU <= 4 && !Kind<KIND>::RAG ? 3 : 1) void cell_kernel(BatchArgs a) {
    extern __shared__ __align__(16) char smem[];
    clear_zero_rows<T>(a);
    const int nut = a.Hu / (16 * WU);
    cell_tile<KIND, T, RT, WU, WK>(a, blockIdx.x / nut, blockIdx.x % nut, smem, NoSync{});
}

// ---------------------------------------------------------------------------
// Streamed tile: rows [16*RT*rtile, +16*RT) x units [16*ub, +16) of a batch of
// a kind without a ragged phase, all gates, the reduction split over WK waves.
// No operand passes through LDS: every lane loads its own MFMA fragments, 16
// bytes of one operand row (gathered through the segment's row list exactly
// as the staged tile gathers) and 16 bytes of a weight block, straight into a
// ring of PD k-groups, so the matrix cores start when the first k-group has
// arrived instead of after the whole A tile.  With the reduction split over
// the waves, no two waves of a work-group read the same operand byte, which is
// all that staging through LDS would have shared.  Each accumulator adds its
// k-groups in ascending order with the same instructions, and the partial sums
// of the waves are added in wave order, as in cell_tile<KIND, T, RT, 1, WK>:
// the two tiles give bitwise equal results.

// Ring of PD k-groups: A fragments of the wave's RT row blocks, weight
// fragments of its G gates.
template <int G, int RT, int PD>
struct SRing {
    uint4 a[PD][RT];
    uint4 b[PD][G];
};

// Operand loads of one k-group: this lane's 16 bytes of each row block's
// operand row in segment s, element columns c + 4 or 8 * (lane / 16) (zero
// past the valid width of the segment, E or H, and for rows whose offset is
// out of range).
template <typename T, int RT, int NSEG, bool HX>
__device__ __forceinline__ void stream_load_a(uint4 (&av)[RT], const u32x4 (&soff)[RT],
                                              __amdgpu_buffer_rsrc_t rx, __amdgpu_buffer_rsrc_t rh, int s, int c,
                                              int E, int H, int lane) {
    constexpr uint32_t OOB = 0x80000000u;
    const bool xs = HX && s == 0;
    const int col = c + (lane >> 4) * Elem<T>::VEC;
    const bool ok = col < (xs ? E : H);
    const __amdgpu_buffer_rsrc_t r = xs ? rx : rh;
#pragma unroll
    for (int rb = 0; rb < RT; ++rb) {
        // a vector value: the compiler picks the segment with selects in
        // registers (as an array it kept the offsets in scratch memory)
        const uint32_t base = NSEG == 1 ? soff[rb][0] : soff[rb][s];
        av[rb] = bload(r, ok ? base + (uint32_t)col * (uint32_t)sizeof(T) : OOB);
    }
}

// Advance the load cursor (k-group lk in segment ls at element lc) by one
// k-group, holding it at the last k-group kg1 - 1 (loads past the end repeat
// it).  Uniform values, no branches.
template <int KG, bool HX>
__device__ __forceinline__ void stream_next(int& lk, int& ls, int& lc, int kg1, int Ep, int Hk) {
    const bool more = lk + 1 < kg1;
    const int nc = lc + KG;
    const bool wrap = nc >= ((HX && ls == 0) ? Ep : Hk);
    lk = more ? lk + 1 : lk;
    ls = more && wrap ? ls + 1 : ls;
    lc = more ? (wrap ? 0 : nc) : lc;
}

template <int KIND, typename T, int RT, int WK>
__device__ __forceinline__ void stream_tile(const BatchArgs& a, int rtile, int ub, char* smem) {
    using KT = Kind<KIND>;
    static_assert(!KT::RAG, "kinds with a ragged phase stage their child rows in LDS");
    constexpr int G = KT::G, NFX = KT::NFIX;
    constexpr bool HX = KT::X;
    constexpr int NSEG = (HX ? 1 : 0) + NFX;
    constexpr int NT = 64 * WK, TM = 16 * RT, TU = 16;
    constexpr int KG = Elem<T>::KG;
    constexpr int NITEM = TM * TU, NI = (NITEM + NT - 1) / NT;
    constexpr int PD = WK >= 16 ? 2 : ring_depth<G>();
    constexpr uint32_t OOB = 0x80000000u;
    constexpr uint32_t ES = sizeof(T);

    float* Z = reinterpret_cast<float*>(smem);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wk = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int row0 = rtile * TM, u0 = ub * TU;
    const int nrows = min(TM, a.m - row0);
    const int nkg = a.K / KG;
    const int kg0 = (nkg * wk) / WK, kg1 = (nkg * (wk + 1)) / WK;

    // ---- 1. row indices, all loads issued at once without branches: this
    // lane's operand rows, the epilogue's result rows and child rows ----
    int srow[NSEG][RT];
#pragma unroll
    for (int rb = 0; rb < RT; ++rb) {
        const int rr = row0 + rb * 16 + (lane & 15);
        int s = 0;
        if constexpr (HX) srow[s++][rb] = seg_row_nb(a.x, rr, a.m);
#pragma unroll
        for (int p = 0; p < NFX; ++p) srow[s++][rb] = seg_row_nb(a.fix[p], rr, a.m);
    }
    int rres[NI], crow[NI][NFX > 0 ? NFX : 1];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int rr = row0 + (tid + NT * q) / TU;
        rres[q] = seg_row_nb(a.res, rr, a.m);
#pragma unroll
        for (int p = 0; p < NFX; ++p) crow[q][p] = seg_row_nb(a.fix[p], rr, a.m);
    }

    // ---- 2. the first PD k-groups: per slot its weights, then its operands
    // (the order of the steady state, so that the loop's waits count the same
    // loads behind each slot on entry as on the back edge).  The loads are
    // unconditional (a wave without k-groups loads k-group 0 and does not use
    // it): with no branch between the index loads and their use, the wait for
    // the indices before the first operand load leaves the weights in flight.
    // Operand byte offsets are out of range, i.e. zero, past the batch and for
    // absent lists ----
    const uint4* Bw = reinterpret_cast<const uint4*>(a.W) + ((size_t)ub * G * nkg) * 64 + lane;
    SRing<G, RT, PD> ring;
    const int xkg = HX ? a.Ep / KG : 0, hkg = a.Hk / KG;
    int lk = kg0, ls, lc;   // load cursor: k-group, its segment, its first element there
    if (kg0 < xkg) {
        ls = 0;
        lc = kg0 * KG;
    } else {
        const int t = kg0 - xkg, p = t / hkg;
        ls = (HX ? 1 : 0) + p;
        lc = (t - p * hkg) * KG;
    }
    // slot 0's weights go out before the operand offsets wait for the indices
    load_b<G>(ring.b[0], Bw, nkg, min(max(lk, 0), nkg - 1));
    __builtin_amdgcn_sched_barrier(0);
    static_assert(NSEG <= 4, "segment offsets are held in a 4-wide vector");
    u32x4 soff[RT];
#pragma unroll
    for (int rb = 0; rb < RT; ++rb) {
        const bool ok = rb * 16 + (lane & 15) < nrows;
        soff[rb] = u32x4{OOB, OOB, OOB, OOB};
        int s = 0;
        if constexpr (HX) {
            soff[rb][s] = ok ? (uint32_t)srow[s][rb] * (uint32_t)a.E * ES : OOB;
            ++s;
        }
#pragma unroll
        for (int p = 0; p < NFX; ++p, ++s)
            soff[rb][s] = ok && a.fix[p].kind != S_NONE ? (uint32_t)srow[s][rb] * (uint32_t)a.H * ES : OOB;
    }
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.xmat, HX ? (uint32_t)a.n_xrows * (uint32_t)a.E * ES : 0u);
    const __amdgpu_buffer_rsrc_t rh = make_rsrc(a.arena_h, (uint32_t)a.n_slots * (uint32_t)a.H * ES);
#pragma unroll
    for (int p = 0; p < PD; ++p) {
        if (p > 0) load_b<G>(ring.b[p], Bw, nkg, min(max(lk, 0), nkg - 1));
        stream_load_a<T, RT, NSEG, HX>(ring.a[p], soff, rx, rh, ls, lc, a.E, a.H, lane);
        stream_next<KG, HX>(lk, ls, lc, kg1, a.Ep, a.Hk);
        __builtin_amdgcn_sched_barrier(0);
    }

    // ---- 3. bias and the children's cell states for the epilogue ----
    float bz[NI][G];   // the packed bias is zero-padded to Hu
#pragma unroll
    for (int q = 0; q < NI; ++q)
#pragma unroll
        for (int g = 0; g < G; ++g) bz[q][g] = a.bias[g * a.Hu + u0 + (tid + NT * q) % TU];
    const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.arena_c, (uint32_t)a.n_slots * (uint32_t)a.H * 4u);
    float cpre[NI][NFX > 0 ? NFX : 1];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + NT * q, r = it / TU, j = u0 + it % TU;
        const bool ok = it < NITEM && r < nrows && j < a.H;
#pragma unroll
        for (int p = 0; p < (NFX > 0 ? NFX : 1); ++p)
            cpre[q][p] = __uint_as_float(bload32(
                rc, NFX > p && reads_child_c<KIND>() && ok && a.fix[p].kind != S_NONE
                        ? ((uint32_t)crow[q][p] * (uint32_t)a.H + (uint32_t)j) * 4u
                        : OOB));
    }

    // ---- 4. gate GEMM over k-groups [kg0, kg1), the ring refilled PD ahead ----
    v4f acc[G][RT];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) acc[g][rt] = v4f{0.f, 0.f, 0.f, 0.f};
    // Each slot's refill is issued right after its matrix-core work and pinned
    // there (scheduling barrier): left alone, the compiler sinks all refills
    // to the end of the unrolled body, and the next iteration then waits for
    // loads it has only just issued.
    int kg = kg0;
    for (; kg + PD < kg1; kg += PD) {
#pragma unroll
        for (int p = 0; p < PD; ++p) {
            kgroup_mma<T, G, RT>(acc, ring.a[p], ring.b[p]);
            load_b<G>(ring.b[p], Bw, nkg, lk);
            stream_load_a<T, RT, NSEG, HX>(ring.a[p], soff, rx, rh, ls, lc, a.E, a.H, lane);
            stream_next<KG, HX>(lk, ls, lc, kg1, a.Ep, a.Hk);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
#pragma unroll
    for (int p = 0; p < PD; ++p)
        if (kg + p < kg1) kgroup_mma<T, G, RT>(acc, ring.a[p], ring.b[p]);
    // partial sums -> Z[wk][row][g][unit] (Z has the LDS to itself)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = rt * 16 + (lane >> 4) * 4 + i;
                Z[((wk * TM + r) * G + g) * TU + (lane & 15)] = acc[g][rt][i];
            }
    __syncthreads();

    // ---- 5. gate pre-activations (partial sums in wave order), epilogue, scatter ----
    T* Hout = reinterpret_cast<T*>(a.arena_h);
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + NT * q, r = it / TU, u = it % TU;
        const int j = u0 + u;
        if (it >= NITEM || r >= nrows || j >= a.H) continue;
        float z[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < WK; ++w) sum += Z[((w * TM + r) * G + g) * TU + u];
            z[g] = sum + bz[q][g];
        }
        float c, h;
        cell_update<KIND>(z, cpre[q], 0.f, 0.f, 0, c, h);
        const size_t o = (size_t)rres[q] * a.H + j;
        a.arena_c[o] = c;
        Hout[o] = from_f<T>(h);
    }
}

template <int KIND, typename T, int RT, int WK>
__host__ __device__ constexpr int stream_lds_bytes() {
    return WK * 16 * RT * Kind<KIND>::G * 16 * 4;
}

// Work-group -> tile in XCD-aware order: work-groups are dispatched round-robin
// over the 8 XCDs, and each XCD takes a contiguous range of tiles, row tiles
// fastest, so the work-groups of a unit block (its weights) share one XCD's L2.
// The grid is a multiple of 8; surplus work-groups exit at once.
template <int KIND, typename T, int RT, int WK>
__global__ __launch_bounds__(64 * WK, WK == 4 ? 3 : 1) void stream_kernel(BatchArgs a) {
    extern __shared__ __align__(16) char smem[];
    const int nut = a.Hu / 16;
    const int nrt = (a.m + 16 * RT - 1) / (16 * RT);
    const int ntile = nrt * nut;
    const int per = (ntile + 7) / 8;
    const int t = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    clear_zero_rows<T>(a);
    if (t >= ntile) return;
    stream_tile<KIND, T, RT, WK>(a, t % nrt, t / nrt, smem);
}

// ---------------------------------------------------------------------------
// Dataflow launch: one persistent launch runs a run of consecutive batches.
// Tiles (batch, row tile, unit tile) are claimed from a global ticket in
// schedule order; a tile waits only for the row tiles that produce its own
// operand rows (every unit tile of each such row tile has signalled), so
// tiles of successive batches overlap.  A claimed tile waits only on tiles
// with smaller tickets, which are held by running work-groups or finished, so
// the launch always drains.  Waits are bounded in time: past `spin_us` the
// tile sets the error flag and proceeds, and every later ticket exits at once.

// Pointer-free description of one batch, resident in device memory.
struct BatchDesc {
    int kind, type, m, H, Hk, Hu, E, Ep, K;
    int x_staged;                 // x rows come from the staged buffer
    int seg_kind[5];              // x, child 0, child 1, ragged, result
    int seg_base[5];
    int seg_off[5];               // offset of the index list in the int buffer, -1 if none
    int rptr_off;                 // ragged row offsets, -1 if none
    int off_b, off_Wr, off_br;    // byte offsets inside the type's packed weights
};

constexpr int FLOW_MAX_TYPES = 16;

struct FlowArgs {
    const int* ibuf;              // descriptor ints
    const BatchDesc* desc;        // per batch of the run
    const int4* tiles;            // {batch, row tile, unit tile, row-tile id}
    const int2* rt_deps;          // per row-tile id: {first dependency, count}
    const int* deps;              // producer row-tile ids
    int* ticket;
    int* error;
    int* done;                    // per row-tile id: unit tiles finished
    int n_tiles, need, spin_us;   // spin_us: bound of one tile's wait, microseconds
    int n_slots, n_xrows;         // arena rows; rows of the x matrix the descriptors address
    const void* x;
    const void* xstaged;
    void* arena_h;
    float* arena_c;
    const void* w[FLOW_MAX_TYPES];
};

__device__ __forceinline__ Seg desc_seg(const BatchDesc& d, const int* ibuf, int i) {
    return Seg{d.seg_kind[i], d.seg_base[i], d.seg_off[i] >= 0 ? ibuf + d.seg_off[i] : nullptr};
}

__device__ __forceinline__ BatchArgs resolve(const BatchDesc& d, const FlowArgs& f) {
    BatchArgs a{};
    a.kind = d.kind;
    a.m = d.m;
    a.H = d.H;
    a.Hk = d.Hk;
    a.Hu = d.Hu;
    a.E = d.E;
    a.Ep = d.Ep;
    a.K = d.K;
    a.x = desc_seg(d, f.ibuf, 0);
    a.fix[0] = desc_seg(d, f.ibuf, 1);
    a.fix[1] = desc_seg(d, f.ibuf, 2);
    a.rag = desc_seg(d, f.ibuf, 3);
    a.res = desc_seg(d, f.ibuf, 4);
    a.rag_ptr = d.rptr_off >= 0 ? f.ibuf + d.rptr_off : nullptr;
    a.xmat = d.x_staged ? f.xstaged : f.x;
    const uint8_t* wb = reinterpret_cast<const uint8_t*>(f.w[d.type]);
    a.W = wb;
    a.bias = reinterpret_cast<const float*>(wb + d.off_b);
    a.Wr = wb + d.off_Wr;
    a.br = reinterpret_cast<const float*>(wb + d.off_br);
    a.arena_h = f.arena_h;
    a.arena_c = f.arena_c;
    a.n_slots = f.n_slots;        // the buffer resources of the tile loads are sized by these
    a.n_xrows = f.n_xrows;
    a.fc = nullptr;               // only child-sum batches on the large tile use it (never in a run)
    return a;
}

struct FlowSync {
    const int2* rt_deps;
    const int* deps;
    int* done;
    int* error;
    int rt, need, spin_us;

    // Thread 0 polls each producer row tile with relaxed atomic loads (coherent
    // across XCDs, no cache maintenance per poll), then issues one acquire
    // fence (agent scope) so that the operand rows read after the barrier are
    // the producers' values.  The wait is bounded in real time: past
    // `spin_us` microseconds (s_memrealtime runs at 100 MHz) it sets the
    // error flag and proceeds; a set error flag ends every other wait.
    __device__ __forceinline__ void wait() const {
        if (threadIdx.x == 0) {
            const int2 di = rt_deps[rt];
            if (di.y > 0) {
                const unsigned long long t0 = wall_clock64();
                const unsigned long long lim = (unsigned long long)spin_us * 100ull;
                bool stop = false;
                for (int k = 0; k < di.y && !stop; ++k) {
                    const int* c = done + deps[di.x + k];
                    int n = 0;
                    while (__hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < need) {
                        __builtin_amdgcn_s_sleep(2);
                        if (wall_clock64() - t0 > lim) {
                            __hip_atomic_store(error, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            stop = true;
                            break;
                        }
                        if ((++n & 63) == 0 && __hip_atomic_load(error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                            stop = true;
                            break;
                        }
                    }
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            }
        }
        __syncthreads();
    }
    // Every wave waits for its own h and c stores, then thread 0 publishes
    // the tile with a release increment (agent scope).
    __device__ __forceinline__ void signal() const {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_fetch_add(done + rt, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
};

// Tile shape of dataflow launches: 16 rows x 16 units, 4 waves splitting K.
constexpr int FLOW_RT = 1, FLOW_WU = 1, FLOW_WK = 4;

template <typename T>
__global__ __launch_bounds__(256) void flow_kernel(FlowArgs f) {
    extern __shared__ __align__(16) char smem[];
    __shared__ int s_ticket;
    for (;;) {
        if (threadIdx.x == 0) {
            int t = __hip_atomic_fetch_add(f.ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__hip_atomic_load(f.error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) t = f.n_tiles;
            s_ticket = t;
        }
        __syncthreads();
        const int t = s_ticket;
        if (t >= f.n_tiles) break;
        const int4 tl = f.tiles[t];
        const BatchArgs a = resolve(f.desc[tl.x], f);
        const FlowSync sync{f.rt_deps, f.deps, f.done, f.error, tl.w, f.need, f.spin_us};
        // every tile body contains barriers, so s_ticket is not rewritten
        // before all threads have read it
        switch (a.kind) {
            case K_CHAIN: cell_tile<K_CHAIN, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_NARY_LEAF: cell_tile<K_NARY_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_NARY_INT: cell_tile<K_NARY_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_GRID: cell_tile<K_GRID, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_CS_LEAF: cell_tile<K_CS_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_CS_INT: cell_tile<K_CS_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_LAT_CHAR: cell_tile<K_LAT_CHAR, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_GRU_LEAF: cell_tile<K_GRU_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            case K_GRU_INT: cell_tile<K_GRU_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
            default: cell_tile<K_LAT_WORD, T, FLOW_RT, FLOW_WU, FLOW_WK>(a, tl.y, tl.z, smem, sync); break;
        }
    }
}

// x staging (the input rows of every batch made contiguous in batch order)
// and clearing of the arena's zero row and pad rows.  Each work-group handles
// 4 rows with one wave per row.
//   rows [0, n_x): xs[i] = x[src[i]]          (row length E elements of T)
//   rows [n_x, n_x + n_zero): arena row zrow[i] of h and c set to zero
//   work-group 0 also clears the `nint` dataflow counters at `ints`
template <typename T>
__global__ __launch_bounds__(256) void stage_kernel(const T* __restrict__ x, T* __restrict__ xs,
                                                    const int* __restrict__ src, int n_x, int E,
                                                    const int* __restrict__ zrow, int n_zero,
                                                    T* __restrict__ arena_h, float* __restrict__ arena_c,
                                                    int H, int* __restrict__ ints, int nint) {
    constexpr int V = Elem<T>::VEC;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nint; i += blockDim.x) ints[i] = 0;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row < n_x) {
        const uint4* s = reinterpret_cast<const uint4*>(x + (size_t)src[row] * E);
        uint4* d = reinterpret_cast<uint4*>(xs + (size_t)row * E);
        for (int c = lane; c < E / V; c += 64) d[c] = s[c];
    } else if (row < n_x + n_zero) {
        const int z = zrow[row - n_x];
        uint4* dh = reinterpret_cast<uint4*>(arena_h + (size_t)z * H);
        for (int c = lane; c < H / V; c += 64) dh[c] = make_uint4(0, 0, 0, 0);
        float4* dc = reinterpret_cast<float4*>(arena_c + (size_t)z * H);
        for (int c = lane; c < H / 4; c += 64) dc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

}  // namespace edbk
