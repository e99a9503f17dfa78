// Roofline probes: the matrix-core rate of the MFMA shapes the batch kernels
// use and the device-memory copy rate, measured on the current device.  They
// give measured denominators next to the datasheet peaks.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <string>

#include "edb_internal.h"

using edb::fail;

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

// Each wave issues iters x 8 MFMAs on register operands, as eight independent
// accumulator chains (enough to cover the MFMA latency).  The instructions are
// written as inline assembly with the accumulators tied to fixed AGPRs:
// through the builtin, the compiler kept the bf16 destination apart from its
// accumulator input and copied every accumulator on every iteration.  The
// s_nop block (tied to the accumulators) covers the matrix-core write -> VALU
// read latency before the sums are read; the sums are written out so that
// none of the work is dead.  iters >= 1.
template <bool BF16>
__global__ __launch_bounds__(256) void mfma_probe_kernel(int iters, float* out) {
    const int t = threadIdx.x;
    v4f c0{0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0, c4 = c0, c5 = c0, c6 = c0, c7 = c0;
    int it = iters;
    if constexpr (BF16) {
        v8bf a, b;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[i] = (__bf16)(0.125f * (float)((t + i) & 7));
            b[i] = (__bf16)(0.0625f * (float)((t * 3 + i) & 15));
        }
        do {
#define EDB_MFMA(c) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b))
            EDB_MFMA(c0); EDB_MFMA(c1); EDB_MFMA(c2); EDB_MFMA(c3);
            EDB_MFMA(c4); EDB_MFMA(c5); EDB_MFMA(c6); EDB_MFMA(c7);
#undef EDB_MFMA
        } while (--it > 0);
    } else {
        const float a = 0.125f * (float)(t & 7), b = 0.0625f * (float)((t * 3) & 15);
        do {
#define EDB_MFMA(c) asm volatile("v_mfma_f32_16x16x4_f32 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b))
            EDB_MFMA(c0); EDB_MFMA(c1); EDB_MFMA(c2); EDB_MFMA(c3);
            EDB_MFMA(c4); EDB_MFMA(c5); EDB_MFMA(c6); EDB_MFMA(c7);
#undef EDB_MFMA
        } while (--it > 0);
    }
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(c0), "+a"(c1), "+a"(c2), "+a"(c3), "+a"(c4), "+a"(c5), "+a"(c6), "+a"(c7));
    const v4f s = c0 + c1 + c2 + c3 + c4 + c5 + c6 + c7;
    out[(int64_t)blockIdx.x * 256 + t] = s[0] + s[1] + s[2] + s[3];
}

// Grid-stride copy of n16 16-byte words, four loads in flight per thread,
// with nontemporal loads and stores (streamed data: on 1 GiB this copies
// about 10% faster than plain accesses).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void copy_probe_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                         int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 v0 = __builtin_nontemporal_load(src + i), v1 = __builtin_nontemporal_load(src + i + stride),
                    v2 = __builtin_nontemporal_load(src + i + 2 * stride),
                    v3 = __builtin_nontemporal_load(src + i + 3 * stride);
        __builtin_nontemporal_store(v0, dst + i);
        __builtin_nontemporal_store(v1, dst + i + stride);
        __builtin_nontemporal_store(v2, dst + i + 2 * stride);
        __builtin_nontemporal_store(v3, dst + i + 3 * stride);
    }
    for (; i < n16; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

edb_status timed(const char* who, hipStream_t st, hipEvent_t e0, hipEvent_t e1, float* ms) {
    hipError_t he = hipGetLastError();
    if (he == hipSuccess) he = hipEventSynchronize(e1);
    if (he == hipSuccess) he = hipEventElapsedTime(ms, e0, e1);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    (void)st;
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string(who) + ": " + hipGetErrorString(he));
    edb::clear_error();
    return EDB_OK;
}

edb_status make_events(const char* who, hipEvent_t* e0, hipEvent_t* e1) {
    *e0 = *e1 = nullptr;
    hipError_t he = hipEventCreate(e0);
    if (he == hipSuccess) he = hipEventCreate(e1);
    if (he != hipSuccess) {
        if (*e0) (void)hipEventDestroy(*e0);
        return fail(EDB_ERR_HIP, std::string(who) + ": " + hipGetErrorString(he));
    }
    return EDB_OK;
}

}  // namespace

extern "C" edb_status edb_probe_mfma(int32_t dtype, int32_t n_workgroups, int32_t iters, float* out, void* stream,
                                     float* ms) {
    if (!out || !ms) return fail(EDB_ERR_INVALID, "edb_probe_mfma: NULL argument");
    if (dtype != EDB_F32 && dtype != EDB_BF16) return fail(EDB_ERR_INVALID, "edb_probe_mfma: dtype must be F32 or BF16");
    if (n_workgroups < 1 || n_workgroups > (1 << 20) || iters < 1 || iters > (1 << 24))
        return fail(EDB_ERR_INVALID, "edb_probe_mfma: n_workgroups in [1, 2^20] and iters in [1, 2^24]");
    if (reinterpret_cast<uintptr_t>(out) & 3u) return fail(EDB_ERR_INVALID, "edb_probe_mfma: out must be 4-byte aligned");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    hipEvent_t e0, e1;
    if (edb_status s = make_events("edb_probe_mfma", &e0, &e1)) return s;
    if (dtype == EDB_BF16)
        hipExtLaunchKernelGGL(mfma_probe_kernel<true>, dim3(n_workgroups), dim3(256), 0, st, e0, e1, 0, iters, out);
    else
        hipExtLaunchKernelGGL(mfma_probe_kernel<false>, dim3(n_workgroups), dim3(256), 0, st, e0, e1, 0, iters, out);
    return timed("edb_probe_mfma", st, e0, e1, ms);
}

extern "C" edb_status edb_probe_copy(const void* src, void* dst, int64_t bytes, int32_t n_workgroups, void* stream,
                                     float* ms) {
    if (!src || !dst || !ms) return fail(EDB_ERR_INVALID, "edb_probe_copy: NULL argument");
    if (bytes < 16 || (bytes & 15) || ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15u))
        return fail(EDB_ERR_INVALID, "edb_probe_copy: bytes and both buffers must be 16-byte multiples / aligned");
    if (n_workgroups < 1 || n_workgroups > (1 << 20))
        return fail(EDB_ERR_INVALID, "edb_probe_copy: n_workgroups must be in [1, 2^20]");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    hipEvent_t e0, e1;
    if (edb_status s = make_events("edb_probe_copy", &e0, &e1)) return s;
    hipExtLaunchKernelGGL(copy_probe_kernel, dim3(n_workgroups), dim3(256), 0, st, e0, e1, 0,
                          reinterpret_cast<const u32x4*>(src), reinterpret_cast<u32x4*>(dst), bytes >> 4);
    return timed("edb_probe_copy", st, e0, e1, ms);
}
