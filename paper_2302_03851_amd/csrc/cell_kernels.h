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
// Work decomposition.  A work-group (4 waves) owns TM = 16*RT rows and
// TU = 16*WU hidden units of the batch, all G gates of those units.  The 4
// waves are split WU along units and WK = 4/WU along the reduction (split-K
// inside the work-group; partial sums are combined in LDS in a fixed order, so
// results do not depend on scheduling).  Each wave computes a 16*RT x 16 x G
// block with 16x16 MFMA tiles: v_mfma_f32_16x16x4_f32 (fp32) or
// v_mfma_f32_16x16x32_bf16 (bf16 inputs, fp32 accumulation).
//
// Packed weights (gate-interleaved, zero padded; produced by edb_pack_weights):
//   main  [Hu/16 unit blocks][G gates][K/KG k-groups][64 lanes][16 bytes]
//   lane l of k-group kg holds, for unit u = ub*16 + l%16 of gate g, the KG/4
//   consecutive k values kg*KG + (l/16)*(KG/4) + i.  With KG = 16 (fp32) this
//   is 4 floats; with KG = 32 (bf16) 8 bf16 values.  One 16-byte load per lane
//   is one B operand (bf16) or four (fp32, one per MFMA of the k-group).
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
       K_LAT_CHAR = 6, K_LAT_WORD = 7 };

enum { S_NONE = 0, S_CONTIG = 1, S_INDEXED = 2 };

// One operand list of a batch: entry r lives in row (kind == CONTIG ? base + r : idx[r]).
struct Seg {
    int kind;
    int base;
    const int* idx;
};

struct BatchArgs {
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
};

template <int KIND> struct Kind;
template <> struct Kind<K_CHAIN>    { static constexpr int G = 3 + 1, NFIX = 1; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_NARY_LEAF>{ static constexpr int G = 3,     NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_NARY_INT> { static constexpr int G = 5,     NFIX = 2; static constexpr bool X = false, RAG = false; };
template <> struct Kind<K_GRID>     { static constexpr int G = 5,     NFIX = 2; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_CS_LEAF>  { static constexpr int G = 3,     NFIX = 0; static constexpr bool X = true,  RAG = false; };
template <> struct Kind<K_CS_INT>   { static constexpr int G = 3,     NFIX = 0; static constexpr bool X = false, RAG = true;  };
template <> struct Kind<K_LAT_CHAR> { static constexpr int G = 5,     NFIX = 1; static constexpr bool X = true,  RAG = true;  };
template <> struct Kind<K_LAT_WORD> { static constexpr int G = 3,     NFIX = 1; static constexpr bool X = true,  RAG = false; };

template <typename T> struct Elem;
template <> struct Elem<float>  { static constexpr int KG = 16; static constexpr int VEC = 4; };
template <> struct Elem<__bf16> { static constexpr int KG = 32; static constexpr int VEC = 8; };

// A-tile row padding in elements: 16 bytes, so that the 16 rows read by one
// MFMA operand load start in different LDS banks.
template <typename T> constexpr int a_pad() { return 16 / (int)sizeof(T); }

__device__ __forceinline__ int seg_row(const Seg& s, int r) {
    return s.kind == S_CONTIG ? s.base + r : s.idx[r];
}

__device__ __forceinline__ float sigm(float z) { return 1.0f / (1.0f + __expf(-z)); }
__device__ __forceinline__ float tanh_f(float z) { return tanhf(z); }

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(__bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ __bf16 from_f<__bf16>(float v) { return (__bf16)v; }

// 16-byte vector of T.
template <typename T> struct Vec16 { uint4 u; };

// LDS budget of one work-group (bytes).
template <int KIND, typename T, int RT, int WU>
__host__ __device__ constexpr int lds_a_bytes(int K) {
    return 16 * RT * (K + a_pad<T>()) * (int)sizeof(T);
}
template <int KIND, typename T, int RT, int WU>
__host__ __device__ constexpr int lds_z_bytes() {
    return (4 / WU) * 16 * RT * Kind<KIND>::G * 16 * WU * 4;
}
template <int KIND, typename T, int RT, int WU>
__host__ __device__ constexpr int lds_zr_bytes() {
    return Kind<KIND>::RAG ? (4 / WU) * 16 * RT * 16 * WU * 4 : 0;
}
template <int KIND, typename T, int RT, int WU>
__host__ __device__ constexpr int lds_bytes(int K) {
    return lds_a_bytes<KIND, T, RT, WU>(K) + lds_z_bytes<KIND, T, RT, WU>() +
           lds_zr_bytes<KIND, T, RT, WU>() + 4 * 16 * RT * 4 /* row index cache */;
}

// Stage rows [row0, row0 + TM) of one K segment into the LDS A tile.
// src row stride = width elements; seg_w = padded width; col0 = K offset.
template <typename T, int TM>
__device__ __forceinline__ void stage_rows(T* A, int AS, const int* rows, int nrows, const T* src,
                                           int width, int seg_w, int col0) {
    constexpr int V = Elem<T>::VEC;
    const int nv = seg_w / V;              // 16-byte chunks per row (padded)
    const int nreal = width / V;           // chunks holding data (width % V == 0)
    for (int it = threadIdx.x; it < TM * nv; it += blockDim.x) {
        const int r = it / nv, c = it % nv;
        uint4 val = make_uint4(0, 0, 0, 0);
        if (r < nrows && c < nreal) {
            const int row = rows[r];
            val = *reinterpret_cast<const uint4*>(src + (size_t)row * width + c * V);
        }
        *reinterpret_cast<uint4*>(A + r * AS + col0 + c * V) = val;
    }
}

// Child sum of h rows for child-sum internal nodes: A[r][k] = sum_children h[k].
template <typename T, int TM>
__device__ __forceinline__ void stage_child_sum(T* A, int AS, const BatchArgs& a, int row0, int nrows) {
    constexpr int V = Elem<T>::VEC;
    const T* h = reinterpret_cast<const T*>(a.arena_h);
    const int nv = a.Hk / V, nreal = a.H / V;
    for (int it = threadIdx.x; it < TM * nv; it += blockDim.x) {
        const int r = it / nv, c = it % nv;
        float acc[V];
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = 0.f;
        if (r < nrows && c < nreal) {
            const int e0 = a.rag_ptr[row0 + r], e1 = a.rag_ptr[row0 + r + 1];
            for (int e = e0; e < e1; ++e) {
                const int row = seg_row(a.rag, e);
                uint4 raw = *reinterpret_cast<const uint4*>(h + (size_t)row * a.H + c * V);
                const T* pv = reinterpret_cast<const T*>(&raw);
#pragma unroll
                for (int i = 0; i < V; ++i) acc[i] += to_f(pv[i]);
            }
        }
        uint4 out;
        T* po = reinterpret_cast<T*>(&out);
#pragma unroll
        for (int i = 0; i < V; ++i) po[i] = from_f<T>(acc[i]);
        *reinterpret_cast<uint4*>(A + r * AS + c * V) = out;
    }
}

// GEMM of one wave: acc[g][rt] += A[rt*16 .. +16][kg range] * Wp[ub][g][kg range].
template <typename T, int G, int RT>
__device__ __forceinline__ void wave_gemm(v4f (&acc)[G][RT], const T* A, int AS, const T* Wp, int nkg,
                                          int ub, int kg0, int kg1, int lane) {
    constexpr int KG = Elem<T>::KG;
    const int arow = lane & 15, aq = lane >> 4;
    // each (ub, g, kg) chunk is 64 lanes x 16 bytes
    const uint4* B = reinterpret_cast<const uint4*>(Wp) + ((size_t)ub * G * nkg) * 64 + lane;
    for (int kg = kg0; kg < kg1; ++kg) {
        uint4 av[RT], bv[G];
#pragma unroll
        for (int g = 0; g < G; ++g) bv[g] = B[((size_t)g * nkg + kg) * 64];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            av[rt] = *reinterpret_cast<const uint4*>(A + (rt * 16 + arow) * AS + kg * KG + aq * (KG / 4));
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
}

template <int KIND, typename T, int RT, int WU>
__global__ __launch_bounds__(256) void cell_kernel(BatchArgs a) {
    using KT = Kind<KIND>;
    constexpr int G = KT::G;
    constexpr int TM = 16 * RT, TU = 16 * WU, WK = 4 / WU;
    constexpr int KG = Elem<T>::KG;
    constexpr int AS_PAD = a_pad<T>();
    constexpr int NSEG = (KT::X ? 1 : 0) + KT::NFIX + (KT::RAG ? 1 : 0);

    extern __shared__ __align__(16) char smem[];
    const int AS = a.K + AS_PAD;                           // A row stride (elements)
    T* A = reinterpret_cast<T*>(smem);
    float* Z = reinterpret_cast<float*>(smem + lds_a_bytes<KIND, T, RT, WU>(a.K));
    float* Zr = Z + WK * TM * G * TU;
    int* rowc = reinterpret_cast<int*>(Zr + (KT::RAG ? WK * TM * TU : 0));   // [4][TM]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int nut = a.Hu / TU;
    const int ut = blockIdx.x % nut, rtile = blockIdx.x / nut;
    const int row0 = rtile * TM, u0 = ut * TU;
    const int nrows = min(TM, a.m - row0);

    // ---- 1. operand row indices of this tile (x, child 0, child 1) ----
    if (tid < TM) {
        const int r = tid;
        const bool ok = r < nrows;
        if constexpr (KT::X) rowc[0 * TM + r] = ok ? seg_row(a.x, row0 + r) : 0;
        if constexpr (KT::NFIX >= 1) rowc[1 * TM + r] = (ok && a.fix[0].kind != S_NONE) ? seg_row(a.fix[0], row0 + r) : 0;
        if constexpr (KT::NFIX >= 2) rowc[2 * TM + r] = (ok && a.fix[1].kind != S_NONE) ? seg_row(a.fix[1], row0 + r) : 0;
        rowc[3 * TM + r] = ok ? seg_row(a.res, row0 + r) : 0;
    }
    __syncthreads();

    // ---- 2. stage the A tile: [x | child h ...] or [child sum of h] ----
    {
        int col = 0;
        if constexpr (KT::X) {
            stage_rows<T, TM>(A, AS, rowc, nrows, reinterpret_cast<const T*>(a.xmat), a.E, a.Ep, col);
            col += a.Ep;
        }
        const T* h = reinterpret_cast<const T*>(a.arena_h);
        if constexpr (KT::NFIX >= 1) {
            // an absent operand list reads the zero row 0 (rowc holds 0)
            stage_rows<T, TM>(A, AS, rowc + TM, nrows, h, a.H, a.Hk, col);
            col += a.Hk;
        }
        if constexpr (KT::NFIX >= 2) {
            stage_rows<T, TM>(A, AS, rowc + 2 * TM, nrows, h, a.H, a.Hk, col);
            col += a.Hk;
        }
        if constexpr (KIND == K_CS_INT) stage_child_sum<T, TM>(A, AS, a, row0, nrows);
        (void)NSEG;
    }
    __syncthreads();

    // ---- 3. gate GEMM: wave (wu, wk) -> unit block u0/16 + wu, k-groups of split wk ----
    const int wu = wave % WU, wk = wave / WU;
    const int nkg = a.K / KG;
    const int ub = u0 / 16 + wu;
    {
        v4f acc[G][RT];
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) acc[g][rt] = v4f{0.f, 0.f, 0.f, 0.f};
        const int kg0 = (nkg * wk) / WK, kg1 = (nkg * (wk + 1)) / WK;
        wave_gemm<T, G, RT>(acc, A, AS, reinterpret_cast<const T*>(a.W), nkg, ub, kg0, kg1, lane);
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
    __syncthreads();

    // ---- 4. per-item epilogue state; items (r, u) owned by fixed threads ----
    constexpr int NI = TM * TU / 256;
    float zsum[NI][G];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + 256 * q, r = it / TU, u = it % TU;
        const int j = u0 + u;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float s = 0.f;
#pragma unroll
            for (int w = 0; w < WK; ++w) s += Z[((w * TM + r) * G + g) * TU + u];
            zsum[q][g] = s + a.bias[g * a.Hu + j];
        }
    }

    // ---- 5. ragged phase: per-child GEMM (child-sum U_f, lattice W_lc) ----
    float racc[NI], rden[NI];
#pragma unroll
    for (int q = 0; q < NI; ++q) { racc[q] = 0.f; rden[q] = 0.f; }
    if constexpr (KT::RAG) {
        const int cbeg = a.rag_ptr[row0];
        const int cend = a.rag_ptr[row0 + nrows];
        const int nkgr = a.Hk / KG;
        const T* Rsrc = KIND == K_CS_INT ? reinterpret_cast<const T*>(a.arena_h) : nullptr;
        for (int cb = cbeg; cb < cend; cb += TM) {
            const int cn = min(TM, cend - cb);
            __syncthreads();   // previous chunk's readers of A / Zr are done
            if (tid < TM) rowc[tid] = tid < cn ? seg_row(a.rag, cb + tid) : 0;
            __syncthreads();
            if constexpr (KIND == K_CS_INT) {
                stage_rows<T, TM>(A, a.Hk + AS_PAD, rowc, cn, Rsrc, a.H, a.Hk, 0);
            } else {
                // lattice: the word cell states c_w (fp32) converted to T
                constexpr int V = Elem<T>::VEC;
                const int nv = a.Hk / V, nreal = a.H / V;
                for (int it = tid; it < TM * nv; it += 256) {
                    const int r = it / nv, c = it % nv;
                    uint4 out = make_uint4(0, 0, 0, 0);
                    T* po = reinterpret_cast<T*>(&out);
                    if (r < cn && c < nreal) {
                        const float* src = a.arena_c + (size_t)rowc[r] * a.H + c * V;
#pragma unroll
                        for (int i = 0; i < V; ++i) po[i] = from_f<T>(src[i]);
                    }
                    *reinterpret_cast<uint4*>(A + r * (a.Hk + AS_PAD) + c * V) = out;
                }
            }
            __syncthreads();
            {
                v4f acc[1][RT];
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) acc[0][rt] = v4f{0.f, 0.f, 0.f, 0.f};
                const int kg0 = (nkgr * wk) / WK, kg1 = (nkgr * (wk + 1)) / WK;
                wave_gemm<T, 1, RT>(acc, A, a.Hk + AS_PAD, reinterpret_cast<const T*>(a.Wr), nkgr, ub,
                                    kg0, kg1, lane);
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int r = rt * 16 + (lane >> 4) * 4 + i;
                        const int u = wu * 16 + (lane & 15);
                        Zr[(wk * TM + r) * TU + u] = acc[0][rt][i];
                    }
            }
            __syncthreads();
#pragma unroll
            for (int q = 0; q < NI; ++q) {
                const int it = tid + 256 * q, r = it / TU, u = it % TU;
                const int j = u0 + u;
                if (r < nrows && j < a.H) {
                    const int e0 = max(a.rag_ptr[row0 + r], cb), e1 = min(a.rag_ptr[row0 + r + 1], cb + cn);
                    for (int e = e0; e < e1; ++e) {
                        float s = a.br[j];
#pragma unroll
                        for (int w = 0; w < WK; ++w) s += Zr[(w * TM + (e - cb)) * TU + u];
                        const float cw = a.arena_c[(size_t)rowc[e - cb] * a.H + j];
                        if constexpr (KIND == K_CS_INT) {
                            racc[q] += sigm(s) * cw;           // f_k * c_k
                        } else {
                            const float l = sigm(zsum[q][4] + s);  // link gate of word k
                            const float ek = __expf(l);
                            racc[q] += ek * cw;
                            rden[q] += ek;
                        }
                    }
                }
            }
        }
    }

    // ---- 6. gate epilogue and scatter of h, c ----
    T* Hout = reinterpret_cast<T*>(a.arena_h);
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        const int it = tid + 256 * q, r = it / TU, u = it % TU;
        const int j = u0 + u;
        if (r >= nrows || j >= a.H) continue;
        const float* z = zsum[q];
        float c, h;
        if constexpr (KIND == K_CHAIN) {
            const float cp = a.fix[0].kind != S_NONE ? a.arena_c[(size_t)rowc[TM + r] * a.H + j] : 0.f;
            c = sigm(z[1]) * cp + sigm(z[0]) * tanh_f(z[2]);
            h = sigm(z[3]) * tanh_f(c);
        } else if constexpr (KIND == K_NARY_LEAF || KIND == K_CS_LEAF) {
            c = sigm(z[0]) * tanh_f(z[2]);
            h = sigm(z[1]) * tanh_f(c);
        } else if constexpr (KIND == K_NARY_INT || KIND == K_GRID) {
            const float c0 = a.fix[0].kind != S_NONE ? a.arena_c[(size_t)rowc[TM + r] * a.H + j] : 0.f;
            const float c1 = a.fix[1].kind != S_NONE ? a.arena_c[(size_t)rowc[2 * TM + r] * a.H + j] : 0.f;
            c = sigm(z[0]) * tanh_f(z[4]) + sigm(z[1]) * c0 + sigm(z[2]) * c1;
            h = sigm(z[3]) * tanh_f(c);
        } else if constexpr (KIND == K_CS_INT) {
            c = sigm(z[0]) * tanh_f(z[2]) + racc[q];
            h = sigm(z[1]) * tanh_f(c);
        } else if constexpr (KIND == K_LAT_WORD) {
            const float cb = a.fix[0].kind != S_NONE ? a.arena_c[(size_t)rowc[TM + r] * a.H + j] : 0.f;
            c = sigm(z[1]) * cb + sigm(z[0]) * tanh_f(z[2]);
            h = 0.f;
        } else {  // K_LAT_CHAR: gates [i, f, o, u, lx]
            const int nw = a.rag_ptr[row0 + r + 1] - a.rag_ptr[row0 + r];
            if (nw == 0) {
                const float cp = a.fix[0].kind != S_NONE ? a.arena_c[(size_t)rowc[TM + r] * a.H + j] : 0.f;
                c = sigm(z[1]) * cp + sigm(z[0]) * tanh_f(z[3]);
            } else {
                const float e0 = __expf(sigm(z[0]));
                c = (e0 * tanh_f(z[3]) + racc[q]) / (e0 + rden[q]);
            }
            h = sigm(z[2]) * tanh_f(c);
        }
        const size_t o = (size_t)rowc[3 * TM + r] * a.H + j;
        a.arena_c[o] = c;
        Hout[o] = from_f<T>(h);
    }
}

// x staging (the input rows of every batch made contiguous in batch order)
// and clearing of the arena's zero row and pad rows.
//   rows [0, n_x): xs[i] = x[src[i]]          (row length E elements of T)
//   rows [n_x, n_x + n_zero): arena row zrow[i] of h and c set to zero
template <typename T>
__global__ __launch_bounds__(256) void stage_kernel(const T* __restrict__ x, T* __restrict__ xs,
                                                    const int* __restrict__ src, int n_x, int E,
                                                    const int* __restrict__ zrow, int n_zero,
                                                    T* __restrict__ arena_h, float* __restrict__ arena_c,
                                                    int H) {
    constexpr int V = Elem<T>::VEC;
    const int row = blockIdx.x;
    if (row < n_x) {
        const uint4* s = reinterpret_cast<const uint4*>(x + (size_t)src[row] * E);
        uint4* d = reinterpret_cast<uint4*>(xs + (size_t)row * E);
        for (int c = threadIdx.x; c < E / V; c += blockDim.x) d[c] = s[c];
    } else if (row < n_x + n_zero) {
        const int z = zrow[row - n_x];
        uint4* dh = reinterpret_cast<uint4*>(arena_h + (size_t)z * H);
        for (int c = threadIdx.x; c < H / V; c += blockDim.x) dh[c] = make_uint4(0, 0, 0, 0);
        float4* dc = reinterpret_cast<float4*>(arena_c + (size_t)z * H);
        for (int c = threadIdx.x; c < H / 4; c += blockDim.x) dc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

}  // namespace edbk
