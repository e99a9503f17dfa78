// Weight-stationary tile for the largest batches of x-only cells (bf16).
//
// A leaf batch of a large mini-batch (every leaf of every tree under
// Algorithm 1) is one GEMM of tens of thousands of gathered x rows by the
// cell's gate matrix.  The large tile re-reads a unit block's weights for
// every row tile; here a work-group owns 32 hidden units (two blocks of 16)
// for the whole launch, holds their weights for all G gates and the whole
// reduction in LDS (G * K / 16 KB), and walks its row tiles of 256 rows in
// turn.  Each of its 8 waves (two per SIMD, so that one wave's gate epilogue
// overlaps the other's matrix-core work) owns 32 rows of a tile: it loads its
// own rows' operand pieces straight from the gathered x rows into a ring of D
// k-groups (16 bytes a lane, row-contiguous) and permutes each into the MFMA
// lane layout one step before use, so the loop shares nothing between waves
// but the read-only weights and needs no barrier.  The ring runs across row
// tiles: the last refills of a tile fetch the next tile's first k-groups,
// which are in flight while the tile's epilogue runs.
//
// The work-group's row table (each row's x offset and result row, for all of
// its tiles) is read once into LDS next to the weights, so the loop issues no
// index loads and its only vector-memory operations are the ring's loads and
// the epilogue's stores.
//
// Each accumulator adds its k-groups in ascending order with
// v_mfma_f32_16x16x32_bf16, and the epilogue adds the bias and applies the
// cell update as the large tile does, so the results are bitwise equal to the
// large tile's.
//
// The epilogue passes each wave's c and h rows through a staging tile of its
// own in LDS, so that every lane stores whole 16-byte pieces of the rows.
//
// On MI355X the LDS pipe bounds the loop: the weight reads and the lane
// permutation share it, over about as much matrix-core time again.  Loaded
// straight in the MFMA lane layout (four rows in each group of four lanes)
// the operands made the launch a quarter slower than the row-contiguous loads
// and permutation below.  The epilogue (gate nonlinearities and the stores,
// which each tile start waits for) adds the rest.
//
// Work-groups are dispatched round-robin over the 8 XCDs; they are numbered
// so that the work-groups of one row group (all unit tiles of the same rows)
// run on one XCD and share those rows in its L2.
#pragma once

#include "big_tile.h"
#include "cell_kernels.h"

namespace edbk {

constexpr int WS_W = 8;                 // waves per work-group
constexpr int WS_NT = 64 * WS_W;        // threads per work-group
constexpr int WS_RB = 2;                // row blocks of 16 per wave
constexpr int WS_TM = WS_W * 16 * WS_RB;   // rows per row tile
constexpr int WS_UB = 2;                // unit blocks of 16 per work-group
constexpr int WS_TU = 16 * WS_UB;       // units per work-group
constexpr int WS_D = 4;                 // k-groups of operands in flight per wave
constexpr int WS_MAXT = 8;              // row tiles per work-group (the row table's capacity)
constexpr int WS_RW = 16 * WS_RB;       // rows per wave
constexpr int WS_CST = WS_TU * 4 + 16;  // staging row stride (bytes) for c (fp32, 16 bytes of padding)
constexpr int WS_HST = WS_TU * 2 + 16;  // staging row stride (bytes) for h (bf16, 16 bytes of padding)
constexpr int WS_STAGE = WS_RW * WS_CST;   // one wave's staging tile (c, then h in the same bytes)

// Kinds the tile serves: x is the only operand (no child lists, no ragged
// phase) and the update reads no child state.
template <int KIND>
__host__ __device__ constexpr bool ws_kind() {
    return Kind<KIND>::X && Kind<KIND>::NFIX == 0 && !Kind<KIND>::RAG && !sums_children<KIND>() &&
           (KIND == K_NARY_LEAF || KIND == K_CS_LEAF || KIND == K_GRU_LEAF);
}

// LDS: the work-group's weight blocks [WS_UB][G][K / 32][64 lanes][16 bytes],
// then the row table: x byte offsets [WS_MAXT][WS_TM], result rows [WS_MAXT][WS_TM],
// then each wave's staging tile for its results.
__host__ __device__ constexpr int ws_weight_bytes(int G, int K) { return WS_UB * G * (K / 32) * 1024; }
__host__ __device__ constexpr int ws_lds_bytes(int G, int K) {
    return ws_weight_bytes(G, K) + WS_MAXT * WS_TM * 8 + WS_W * WS_STAGE;
}

// grid = (Hu / WS_TU) unit tiles x ngr row groups, ngr a multiple of 8 with
// ceil(m / WS_TM) <= ngr * WS_MAXT; K / 32 a multiple of WS_D and at least
// 2 WS_D, so that a refill targets at most the next row tile.
template <int KIND>
__global__ __launch_bounds__(WS_NT, 1) void ws_kernel(BatchArgs a) {
    static_assert(WS_TM <= WS_NT, "one row of the row table per thread and tile");
    static_assert(WS_RW * 8 % 64 == 0 && WS_RW * 4 % 64 == 0, "whole 16-byte pieces per lane");
    constexpr int G = Kind<KIND>::G;
    constexpr uint32_t OOB = 0x80000000u;
    extern __shared__ __align__(16) char smem[];
    clear_zero_rows<__bf16>(a);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nkg = a.K / 32;
    const int nut = a.Hu / WS_TU;
    const int ngr = (int)gridDim.x / nut;            // row groups (a multiple of 8)
    const int per = (int)gridDim.x / 8;              // work-groups per XCD
    const int flat = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    const int ut = flat % nut, rg = flat / nut;
    const int u0 = ut * WS_TU;
    const int nrt = (a.m + WS_TM - 1) / WS_TM;
    const int ntile = rg < nrt ? min((nrt - 1 - rg) / ngr + 1, WS_MAXT) : 0;   // tiles rg, rg + ngr, ...
    if (ntile == 0) return;

    const int nw = WS_UB * G * nkg;                  // 1 KB weight blocks
    uint32_t* xo_l = reinterpret_cast<uint32_t*>(smem + nw * 1024);
    int* res_l = reinterpret_cast<int*>(xo_l + WS_MAXT * WS_TM);
    char* stg = reinterpret_cast<char*>(res_l + WS_MAXT * WS_TM) + wave * WS_STAGE;   // this wave's staging tile
    {
        // the stationary weights: the two unit blocks' blocks are contiguous in
        // the packed matrix ((unit block * G + gate) * nkg + k-group), copied
        // straight to LDS, 1 KB a wave per copy
        const char* src = reinterpret_cast<const char*>(a.W) + (size_t)(u0 / 16) * G * nkg * 1024;
        const __amdgpu_buffer_rsrc_t rw = make_rsrc(src, (uint32_t)nw * 1024u);
        for (int c = wave; c < nw; c += WS_W) dma16(rw, (uint32_t)c * 1024u + (uint32_t)lane * 16u, smem + c * 1024);
        // the row table; rows past the batch get an out-of-range x offset
        const Seg sx = a.x, sr = a.res;
        const __amdgpu_buffer_rsrc_t rix = make_rsrc(sx.idx, sx.kind == S_INDEXED ? (uint32_t)a.m * 4u : 0u);
        const __amdgpu_buffer_rsrc_t rir = make_rsrc(sr.idx, sr.kind == S_INDEXED ? (uint32_t)a.m * 4u : 0u);
        int vx[WS_MAXT], vr[WS_MAXT];
#pragma unroll
        for (int t = 0; t < WS_MAXT; ++t) {
            const int r = min((rg + t * ngr) * WS_TM + tid, a.m - 1);
            vx[t] = (int)bload32(rix, (uint32_t)r * 4u);
            vr[t] = (int)bload32(rir, (uint32_t)r * 4u);
        }
#pragma unroll
        for (int t = 0; t < WS_MAXT; ++t) {
            const int r = (rg + t * ngr) * WS_TM + tid;
            if (t < ntile && tid < WS_TM) {
                const int x = sx.kind == S_CONTIG ? sx.base + r : vx[t];
                xo_l[t * WS_TM + tid] = r < a.m ? (uint32_t)x * (uint32_t)a.E * 2u : OOB;
                res_l[t * WS_TM + tid] = sr.kind == S_CONTIG ? sr.base + r : vr[t];
            }
        }
    }
    __builtin_amdgcn_s_waitcnt(0);   // the weight copies (LDS-DMA) have landed
    __syncthreads();
    const uint4* Ws = reinterpret_cast<const uint4*>(smem) + lane;

    float bz[WS_UB][G];   // the packed bias is zero-padded to Hu
#pragma unroll
    for (int ub = 0; ub < WS_UB; ++ub)
#pragma unroll
        for (int g = 0; g < G; ++g) bz[ub][g] = a.bias[g * a.Hu + u0 + ub * 16 + (lane & 15)];

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.xmat, (uint32_t)a.n_xrows * (uint32_t)a.E * 2u);
    // The operand rows are loaded row-contiguous: lanes 4j .. 4j + 3 read the
    // 64 bytes of one k-group of row j of a row block (16 bytes each), so each
    // group of four lanes touches one cache line.  (In the MFMA lane layout,
    // lane l holding row l % 16, four lanes in a row touch four lines: the
    // vector L1 then handles four times the accesses per load, and that bound
    // the loop.)  A lane permutation (lane bits rotated by two) then moves
    // each fragment to the MFMA layout.
    const int wrow = wave * WS_RW + (lane >> 2);   // this lane's operand row in a tile (row block 0)
    const int perm = ((((lane & 15) << 2) | (lane >> 4))) * 4;   // byte address of the source lane

    // x offsets of this lane's operand rows in tile t (out of range past the last tile)
    auto offsets = [&](int t, uint32_t (&off)[WS_RB]) {
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb) off[rb] = t < ntile ? xo_l[t * WS_TM + wrow + rb * 16] : OOB;
    };
    // row-contiguous operand pieces of k-group kg: 16 bytes of the lane's row
    // at element kg * 32 + 8 * (lane % 4), zero past E
    auto load_a = [&](uint4 (&av)[WS_RB], const uint32_t (&off)[WS_RB], int kg) {
        const int col = kg * 32 + (lane & 3) * 8;
        const bool ok = col < a.E;
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb) av[rb] = bload(rx, ok ? off[rb] + (uint32_t)col * 2u : OOB);
    };
    // the MFMA fragments: lane l takes the piece of lane 4 (l % 16) + l / 16
    auto permute = [&](const uint4 (&av)[WS_RB], uint4 (&fa)[WS_RB]) {
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb) {
            fa[rb].x = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)av[rb].x);
            fa[rb].y = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)av[rb].y);
            fa[rb].z = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)av[rb].z);
            fa[rb].w = (uint32_t)__builtin_amdgcn_ds_bpermute(perm, (int)av[rb].w);
        }
    };

    v4f acc[WS_UB][G][WS_RB];
    uint4 ring[WS_D][WS_RB];   // row-contiguous pieces of the next WS_D steps
    uint4 fa[2][WS_RB];        // MFMA fragments: this step's, the next step's
    uint4 bfa[WS_UB][G], bfb[WS_UB][G];   // weight fragments: this step's, the next step's
    auto read_b = [&](uint4 (&bf)[WS_UB][G], int kg) {
#pragma unroll
        for (int ub = 0; ub < WS_UB; ++ub)
#pragma unroll
            for (int g = 0; g < G; ++g) bf[ub][g] = Ws[((ub * G + g) * nkg + kg) * 64];
    };
    uint32_t offc[WS_RB], offn[WS_RB];   // the current and the next row tile
    // the ring slot that holds step kg0 + p + 1 (p + 1 mod WS_D) is permuted into
    // the next step's fragments and refilled with the step WS_D after it,
    // k-group t of the current tile or t - nkg of the next
    auto advance = [&](int q, uint4 (&fn)[WS_RB], int t) {
        permute(ring[q], fn);
        const bool nxt = t >= nkg;
        uint32_t offr[WS_RB];
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb) offr[rb] = nxt ? offn[rb] : offc[rb];
        load_a(ring[q], offr, nxt ? t - nkg : t);
    };
    // one step of k-group kg0 + p: the next step's weight fragments (k-group
    // kgb) are read from LDS and its operand fragments permuted, the ring slot
    // refilled, then this step's MFMAs.  The scheduling barriers keep the
    // reads, the permutation and the refill ahead of the MFMAs (the scheduler
    // would sink every refill to the end of the group, where the next group
    // would wait for all of them).
    auto step = [&](const uint4 (&bfc)[WS_UB][G], uint4 (&bfn)[WS_UB][G], const uint4 (&fc)[WS_RB],
                    uint4 (&fn)[WS_RB], int kg0, int p, int kgb) {
        read_b(bfn, kgb);
        advance((p + 1) % WS_D, fn, kg0 + p + 1 + WS_D);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ub = 0; ub < WS_UB; ++ub)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int rb = 0; rb < WS_RB; ++rb)
                    acc[ub][g][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(v8bf, fc[rb]), __builtin_bit_cast(v8bf, bfc[ub][g]),
                        acc[ub][g][rb], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
    };
    // k-groups kg0 .. kg0 + WS_D - 1 (WS_D even: the weight and operand
    // fragments alternate between two sets each, and the first set holds the
    // next group's first step)
    auto group = [&](int kg0) {
        static_assert(WS_D % 2 == 0, "the fragments alternate between two sets");
#pragma unroll
        for (int p = 0; p < WS_D; p += 2) {
            step(bfa, bfb, fa[0], fa[1], kg0, p, kg0 + p + 1);
            const int kn = kg0 + p + 2;
            step(bfb, bfa, fa[1], fa[0], kg0, p + 1, kn < nkg ? kn : 0);
        }
    };

    offsets(0, offc);
    offsets(1, offn);
#pragma unroll
    for (int p = 0; p < WS_D; ++p) load_a(ring[p], offc, p);
    read_b(bfa, 0);
    advance(0, fa[0], WS_D);   // step 0's fragments; slot 0 refilled with step WS_D
    __bf16* Hout = reinterpret_cast<__bf16*>(a.arena_h);
    for (int i = 0; i < ntile; ++i) {
#pragma unroll
        for (int ub = 0; ub < WS_UB; ++ub)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int rb = 0; rb < WS_RB; ++rb) acc[ub][g][rb] = v4f{0.f, 0.f, 0.f, 0.f};
        // the previous tile's stores are pending with the ring's loads, and the
        // compiler waits for every vector-memory operation where loads and
        // stores are pending together: wait once here (unconditionally, so that
        // no path into the loop carries stores), and the loop waits for the
        // ring slot by slot
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0)
        for (int kg0 = 0; kg0 < nkg; kg0 += WS_D) group(kg0);

        // ---- epilogue of row tile i: bias, gates, cell update, h and c ----
        // The wave's results pass through its staging tile so that every lane
        // stores whole 16-byte pieces of the rows (c: 8 a row, h: 4 a row); H
        // is a multiple of 8, so a piece is either inside the row or past H.
        // The wave's LDS operations run in order, so no wait separates the
        // staging writes from the reads, nor the c reads from the h writes.
        const int base = (rg + i * ngr) * WS_TM + wave * WS_RW;   // the wave's first row
        const int* rres = res_l + i * WS_TM + wave * WS_RW;
        float hv[WS_RB][4][WS_UB];
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int rw = rb * 16 + (lane >> 4) * 4 + q;   // row of the wave
#pragma unroll
                for (int ub = 0; ub < WS_UB; ++ub) {
                    float z[G], cp[1] = {0.f};
#pragma unroll
                    for (int g = 0; g < G; ++g) z[g] = acc[ub][g][rb][q] + bz[ub][g];
                    float c, h;
                    cell_update<KIND>(z, cp, 0.f, 0.f, 0, c, h);
                    *reinterpret_cast<float*>(stg + rw * WS_CST + (ub * 16 + (lane & 15)) * 4) = c;
                    hv[rb][q][ub] = h;
                }
            }
#pragma unroll
        for (int k = 0; k < WS_RW * 8 / 64; ++k) {
            const int e = k * 64 + lane, rw = e >> 3, p = e & 7;
            const float4 v = *reinterpret_cast<const float4*>(stg + rw * WS_CST + p * 16);
            if (base + rw < a.m && u0 + p * 4 < a.H)
                *reinterpret_cast<float4*>(a.arena_c + (size_t)rres[rw] * a.H + u0 + p * 4) = v;
        }
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int ub = 0; ub < WS_UB; ++ub)
                    *reinterpret_cast<__bf16*>(stg + (rb * 16 + (lane >> 4) * 4 + q) * WS_HST +
                                               (ub * 16 + (lane & 15)) * 2) = from_f<__bf16>(hv[rb][q][ub]);
#pragma unroll
        for (int k = 0; k < WS_RW * 4 / 64; ++k) {
            const int e = k * 64 + lane, rw = e >> 2, p = e & 3;
            const uint4 v = *reinterpret_cast<const uint4*>(stg + rw * WS_HST + p * 16);
            if (base + rw < a.m && u0 + p * 8 < a.H)
                *reinterpret_cast<uint4*>(Hout + (size_t)rres[rw] * a.H + u0 + p * 8) = v;
        }
#pragma unroll
        for (int rb = 0; rb < WS_RB; ++rb) offc[rb] = offn[rb];
        offsets(i + 2, offn);
    }
}

}  // namespace edbk
