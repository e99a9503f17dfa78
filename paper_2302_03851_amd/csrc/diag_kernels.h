// Unfused row copies for the split-phase diagnostic.  Section 3.1 prices a
// batch's execution as a gather of its operand rows into one contiguous
// buffer, the batched kernel, and a scatter of its results to where the
// consumers read them.  The fused batch kernels do the gather in their
// prologue and the scatter in their epilogue; these kernels run the two
// copies alone, so that their HBM time can be measured on their own.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "cell_kernels.h"

namespace edbk {

// n rows of row_bytes each: row r is copied from src row srow(r) to dst row
// drow(r) (row strides = row_bytes).  Rows whose index falls outside
// [0, src_rows) or [0, dst_rows) are skipped.
struct CopyStream {
    const char* src;
    char* dst;
    Seg srow, drow;
    int n;
    int row_bytes;   // a multiple of 2
    int64_t src_rows, dst_rows;
};

constexpr int MAX_COPY_STREAMS = 7;   // x, two positional children (h and c), ragged children (h and c)

struct CopyArgs {
    CopyStream s[MAX_COPY_STREAMS];
    int n_streams;
};

__device__ __forceinline__ void copy_row(const CopyStream& s, int r, int lane) {
    const int64_t sr = seg_row(s.srow, r), dr = seg_row(s.drow, r);
    if (sr < 0 || sr >= s.src_rows || dr < 0 || dr >= s.dst_rows) return;
    const char* src = s.src + sr * s.row_bytes;
    char* dst = s.dst + dr * s.row_bytes;
    if ((s.row_bytes & 15) == 0) {
        const uint4* s4 = reinterpret_cast<const uint4*>(src);
        uint4* d4 = reinterpret_cast<uint4*>(dst);
        for (int q = lane; q < (s.row_bytes >> 4); q += 64) d4[q] = s4[q];
    } else {
        const uint16_t* s2 = reinterpret_cast<const uint16_t*>(src);
        uint16_t* d2 = reinterpret_cast<uint16_t*>(dst);
        for (int q = lane; q < (s.row_bytes >> 1); q += 64) d2[q] = s2[q];
    }
}

// Grid: x = groups of 4 rows (one wave per row), y = copy stream.  The stream
// is picked with constant indices (a dynamic index into the argument struct
// would make the compiler copy it to scratch memory).
__global__ __launch_bounds__(256) void copy_rows_kernel(CopyArgs a) {
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    switch (blockIdx.y) {
#define EDB_COPY_CASE(i) \
    case i:              \
        if (i < a.n_streams && r < a.s[i].n) copy_row(a.s[i], r, lane); \
        break;
        EDB_COPY_CASE(0)
        EDB_COPY_CASE(1)
        EDB_COPY_CASE(2)
        EDB_COPY_CASE(3)
        EDB_COPY_CASE(4)
        EDB_COPY_CASE(5)
        EDB_COPY_CASE(6)
#undef EDB_COPY_CASE
        default: break;
    }
}

}  // namespace edbk
