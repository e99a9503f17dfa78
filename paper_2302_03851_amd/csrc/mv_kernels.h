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
// w % 2 (0: B a, 1: A b).  fp32 rows: lane l = 16 g + q loads 16 bytes
// (columns 4q .. 4q+3 of a 64-column block) of weighted row j = 4 i + g, so
// one wave instruction reads four rows; each lane group g accumulates its
// rows in order, and the four groups' sums are added at the end (g 0 + g 1,
// then + (g 2 + g 3)).  H is a multiple of 4 (16-byte rows).
template <typename T>
__global__ __launch_bounds__(256) void mv_matvec_kernel(BatchArgs a, T* __restrict__ u) {
    static_assert(sizeof(T) == 4, "fp32 rows");
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (w >= 2 * a.m) return;
    const int r = w >> 1, half = w & 1, H = a.H;
    const int grp = lane >> 4, q = lane & 15;
    const float* h = reinterpret_cast<const float*>(a.arena_h);
    // half 0: B a (weights: the left vector, rows: the right matrix's columns)
    const int vrow = seg_row(half == 0 ? a.fix[0] : a.fix[1], r);
    const int e0 = a.rag_ptr[r] + (half == 0 ? H : 0);
    const float* vec = h + (size_t)vrow * H;
    float* out = reinterpret_cast<float*>(u) + (size_t)r * 2 * H + (size_t)half * H;
    for (int c0 = 0; c0 < H; c0 += 64) {
        const int c = c0 + 4 * q;
        const int cc = c < H ? c : H - 4;   // lanes past H read a valid chunk, store nothing
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        int j = grp;
        for (; j + 4 < H; j += 8) {   // rows j and j + 4 of this lane group
            const int m0 = seg_row(a.rag, e0 + j), m1 = seg_row(a.rag, e0 + j + 4);
            const float w0 = vec[j], w1 = vec[j + 4];
            const float4 v0 = *reinterpret_cast<const float4*>(h + (size_t)m0 * H + cc);
            const float4 v1 = *reinterpret_cast<const float4*>(h + (size_t)m1 * H + cc);
            acc.x = fmaf(w0, v0.x, acc.x); acc.y = fmaf(w0, v0.y, acc.y);
            acc.z = fmaf(w0, v0.z, acc.z); acc.w = fmaf(w0, v0.w, acc.w);
            acc.x = fmaf(w1, v1.x, acc.x); acc.y = fmaf(w1, v1.y, acc.y);
            acc.z = fmaf(w1, v1.z, acc.z); acc.w = fmaf(w1, v1.w, acc.w);
        }
        for (; j < H; j += 4) {
            const int m0 = seg_row(a.rag, e0 + j);
            const float w0 = vec[j];
            const float4 v0 = *reinterpret_cast<const float4*>(h + (size_t)m0 * H + cc);
            acc.x = fmaf(w0, v0.x, acc.x); acc.y = fmaf(w0, v0.y, acc.y);
            acc.z = fmaf(w0, v0.z, acc.z); acc.w = fmaf(w0, v0.w, acc.w);
        }
        // sum over the four lane groups: (g0 + g1) + (g2 + g3)
        acc.x += __shfl_xor(acc.x, 16); acc.y += __shfl_xor(acc.y, 16);
        acc.z += __shfl_xor(acc.z, 16); acc.w += __shfl_xor(acc.w, 16);
        acc.x += __shfl_xor(acc.x, 32); acc.y += __shfl_xor(acc.y, 32);
        acc.z += __shfl_xor(acc.z, 32); acc.w += __shfl_xor(acc.w, 32);
        if (grp == 0 && c < H) *reinterpret_cast<float4*>(out + c) = acc;
    }
}

}  // namespace edbk
