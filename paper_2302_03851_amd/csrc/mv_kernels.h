// MV-RNN (Table 2): the matrix-vector products of a vector batch.
//
// An MV-RNN node with left child (a, A) and right child (b, B) computes its
// vector from [B a ; A b].  A child's d x d matrix lives in the arena as d
// rows, row j = column j of the matrix, so B a = sum_j a_j * (row j of B) is
// a weighted sum of arena rows.  The vector batch's descriptors give, per
// node, its two vector children (positional lists 0 and 1) and a ragged list
// of exactly 2d entries: the d column rows of A, then the d column rows of B.
// mv_matvec_kernel writes u[r] = [B a, A b] (2d values of T per row); the
// batch's GEMM then reads u as its x operand.
#pragma once

#include <hip/hip_runtime.h>

#include "cell_kernels.h"

namespace edbk {

// Grid: ceil(2 m / 4) work-groups of 4 waves; wave w handles row w / 2, half
// w % 2 (0: B a, 1: A b).  Lane l accumulates columns l, l + 64, ... of the
// half in fp32, over the d weighted rows in order j = 0 .. d-1.
template <typename T>
__global__ __launch_bounds__(256) void mv_matvec_kernel(BatchArgs a, T* __restrict__ u) {
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (w >= 2 * a.m) return;
    const int r = w >> 1, half = w & 1, H = a.H;
    const T* h = reinterpret_cast<const T*>(a.arena_h);
    // half 0: B a (weights: the left vector, rows: the right matrix's columns)
    const int vrow = seg_row(half == 0 ? a.fix[0] : a.fix[1], r);
    const int e0 = a.rag_ptr[r] + (half == 0 ? H : 0);
    const T* vec = h + (size_t)vrow * H;
    T* out = u + (size_t)r * 2 * H + (size_t)half * H;
    for (int c0 = 0; c0 < H; c0 += 64) {
        const int c = c0 + lane;
        const int cc = c < H ? c : H - 1;   // lanes past H read a valid column, store nothing
        float acc = 0.f;
        int j = 0;
        for (; j + 8 <= H; j += 8) {
            int mr[8];
            float wj[8], mv[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) mr[q] = seg_row(a.rag, e0 + j + q);
#pragma unroll
            for (int q = 0; q < 8; ++q) wj[q] = to_f(vec[j + q]);
#pragma unroll
            for (int q = 0; q < 8; ++q) mv[q] = to_f(h[(size_t)mr[q] * H + cc]);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc = fmaf(wj[q], mv[q], acc);
        }
        for (; j < H; ++j) acc = fmaf(to_f(vec[j]), to_f(h[(size_t)seg_row(a.rag, e0 + j) * H + cc]), acc);
        if (c < H) out[c] = from_f<T>(acc);
    }
}

}  // namespace edbk
