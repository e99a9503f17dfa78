// Large-batch tile for cells on gfx950 (bf16 and fp32).
//
// The first batches of a schedule can hold thousands of nodes (all leaves of
// a mini-batch form one batch under Algorithm 1), and there the cell GEMM is a
// dense contraction large enough to be bound by the matrix cores.  This tile
// raises the reuse of every operand fetched from L2: a work-group of 4 waves
// (2 along rows x 2 along units) owns TM = 32*RB rows and TU = 32*CU hidden
// units with all G gates, and both operands pass through LDS in chunks of 128
// bytes of k (64 bf16 or 32 fp32 values), double buffered so that the global
// loads of chunk c+1 are in flight while the matrix cores work on chunk c.
// Each wave holds a 16*RB x 16*CU x G block of accumulators (fp32; bf16 on
// v_mfma_f32_16x16x32_bf16, fp32 on four v_mfma_f32_16x16x4_f32 per 16-byte
// fragment), so the gate epilogue finds all G pre-activations of an element
// in one lane.  A chunk is two k-groups of either type (32 bf16 or 16 fp32
// values: one 1 KB weight block each), so the stages have the same layout.
//
// The operand rows are gathered through the batch's segment descriptors
// exactly as in the small tile (contiguous lists as base + row, indexed lists
// through their slot list), and the k-groups of every accumulator are added
// in ascending order with the same instruction, so a batch computed here is
// bitwise equal to the small tile without split-K.
//
// Work-groups are dispatched round-robin over the 8 XCDs; the tile order is
// remapped so that each XCD owns a contiguous range of tiles, unit tiles
// fastest: the work-groups sharing a row tile's operand rows run on one XCD
// and hit in its L2.
#pragma once

#include "cell_kernels.h"

namespace edbk {

// k values per LDS stage: two k-groups, 128 bytes of each operand row
template <typename T> constexpr int big_bk() { return 128 / (int)sizeof(T); }

// Size classes vb: unit blocks per wave CU (2 for classes 0-2, 1 for 3-4: the
// narrow classes give fp32 batches, whose matrix-core work per byte is eight
// times bf16's, enough work-groups) and row blocks per wave RB (8, 4, 2, 2, 1,
// capped so that the accumulators, 4 * CU * G * RB registers, stay within 192).
constexpr int NUM_BIG_CLASSES = 5;
__host__ __device__ constexpr int big_cu(int vb) { return vb < 3 ? 2 : 1; }
__host__ __device__ constexpr int big_rb(int G, int vb) {
    const int want = vb == 0 ? 8 : vb == 1 ? 4 : vb == 4 ? 1 : 2;
    const int cap = 192 / (4 * big_cu(vb) * G);
    return want < cap ? want : cap;
}

// One LDS stage: A [TM rows][64 k] bf16 (128 bytes a row, 16-byte pieces
// XOR-swizzled by row: piece q of row r sits in slot q ^ (r & 7), so that the
// 16 rows one MFMA operand read touches fall in distinct banks), then the
// weight blocks [2 CU unit blocks][G][2 k-groups][64 lanes][16 bytes].
template <int G, int RB, int CU>
__host__ __device__ constexpr int big_stage_bytes() {
    return 32 * RB * 128 + 2 * CU * G * 2 * 1024;
}
template <int KIND, int VB>
__host__ __device__ constexpr int big_lds_bytes() {   // the same for both element types
    return 2 * big_stage_bytes<Kind<KIND>::G, big_rb(Kind<KIND>::G, VB), big_cu(VB)>();
}

// Direct global -> LDS copy of 16 bytes per lane: lane l's bytes at byte
// offset off land at lds + 16 l (lds is wave-uniform).  Offsets past the end
// of the buffer read as zero.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t off, char* lds) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, off, 0, 0, 0);
}

// Copies of one k chunk into an LDS stage.  The chunk lies in one operand
// segment (uniform sg: 0 = x when the kind has x, then child positions); lane
// column col of that segment's source rows, zero where col >= lim.
template <typename T, int RB, int NSEG, int NBW, bool HAS_X>
__device__ __forceinline__ void big_copy(const uint32_t (&soff)[NSEG][RB], const uint32_t (&woff)[NBW],
                                         __amdgpu_buffer_rsrc_t rx, __amdgpu_buffer_rsrc_t rh,
                                         __amdgpu_buffer_rsrc_t rw, int c, int sg, int col, int lim, char* As,
                                         char* Bs, int wave) {
    constexpr uint32_t OOB = 0x80000000u;
    const bool have = col < lim;
    const bool xs = HAS_X && sg == 0;
#pragma unroll
    for (int j = 0; j < RB; ++j) {
        uint32_t ro = soff[0][j];
#pragma unroll
        for (int s = 1; s < NSEG; ++s)
            if (sg == s) ro = soff[s][j];
        const uint32_t off = have ? ro + (uint32_t)col * (uint32_t)sizeof(T) : OOB;
        if (xs) dma16(rx, off, As + (4 * j + wave) * 1024);
        else dma16(rh, off, As + (4 * j + wave) * 1024);
    }
#pragma unroll
    for (int j = 0; j < NBW; ++j) dma16(rw, woff[j] + (uint32_t)c * 2048u, Bs + (4 * j + wave) * 1024);
}

// k-group pair of one LDS stage on the matrix cores.  Each accumulator adds
// its k-groups in order, and within a fp32 k-group its four k-steps in order,
// as the small tile does.
template <typename T, int RB, int CU, int G>
__device__ __forceinline__ void big_compute(v4f (&acc)[CU][G][RB], const char* As, const uint4* Bs, int wr, int wc,
                                            int lane) {
#pragma unroll
    for (int kgi = 0; kgi < 2; ++kgi) {
        uint4 af[RB], bf[CU][G];
        // row wr*16RB + rb*16 + (lane & 15), piece kgi*4 + lane/16, swizzled by row & 7 = lane & 7
        const int slot = ((kgi * 4 + (lane >> 4)) ^ (lane & 7)) * 16;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
            af[rb] = *reinterpret_cast<const uint4*>(As + (wr * 16 * RB + rb * 16 + (lane & 15)) * 128 + slot);
#pragma unroll
        for (int cu = 0; cu < CU; ++cu)
#pragma unroll
            for (int g = 0; g < G; ++g) bf[cu][g] = Bs[(((wc * CU + cu) * G + g) * 2 + kgi) * 64 + lane];
#pragma unroll
        for (int cu = 0; cu < CU; ++cu)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    if constexpr (sizeof(T) == 2) {
                        acc[cu][g][rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(v8bf, af[rb]), __builtin_bit_cast(v8bf, bf[cu][g]), acc[cu][g][rb], 0,
                            0, 0);
                    } else {
#pragma unroll
                        for (int j = 0; j < 4; ++j)
                            acc[cu][g][rb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                __uint_as_float((&af[rb].x)[j]), __uint_as_float((&bf[cu][g].x)[j]), acc[cu][g][rb], 0,
                                0, 0);
                    }
                }
    }
}

// Rows of cell states the epilogue reads per tile row (copied into the
// stages after the chunk loop): the positional children's, the forget GEMM's
// own children's, the parent GEMM's product sums.  Kinds with none leave the
// stages free during the epilogue.
template <int KIND>
__host__ __device__ constexpr int big_ncr() {
    return (KIND == K_CS_FORGET || KIND == K_CS_PARENT) ? 1 : (reads_child_c<KIND>() ? Kind<KIND>::NFIX : 0);
}

// Byte offsets of one tile's chunk copies (see big_tile): per A copy j the
// source row of each operand segment (OOB: zero), per weight copy j its block.
template <int KIND, typename T, int VB, int NSEG, int RB, int NBW>
__device__ __forceinline__ void big_offsets(const BatchArgs& a, int tile, int wave, int lane,
                                            uint32_t (&soff)[NSEG][RB], uint32_t (&woff)[NBW]) {
    using KT = Kind<KIND>;
    constexpr uint32_t ES = sizeof(T), OOB = 0x80000000u;
    constexpr int G = KT::G, NFX = KT::NFIX, TM = 32 * RB, TU = 32 * big_cu(VB);
    const int nut = a.Hu / TU;
    const int row0 = (tile / nut) * TM, u0 = (tile % nut) * TU;
    const int nrows = min(TM, a.m - row0);
    const int nkg = a.K / Elem<T>::KG;
    // A copies: wave w's j-th copy fills rows (4 j + w) * 8 .. + 8 of the stage
#pragma unroll
    for (int j = 0; j < RB; ++j) {
        const int r = (4 * j + wave) * 8 + (lane >> 3);
        const bool ok = r < nrows;
        int s = 0;
        if constexpr (KT::X) soff[s++][j] = ok ? (uint32_t)seg_row(a.x, row0 + r) * (uint32_t)a.E * ES : OOB;
#pragma unroll
        for (int p = 0; p < NFX; ++p)
            soff[s++][j] = !ok ? OOB
                               : (a.fix[p].kind == S_NONE ? 0u
                                                          : (uint32_t)seg_row(a.fix[p], row0 + r) * (uint32_t)a.H * ES);
    }
    // weight copies: wave w's j-th copy is block b = 4 j + w = ((ubi * G + g) * 2 + kgi)
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
        const int b = 4 * j + wave;
        const int kgi = b & 1, g = (b >> 1) % G, ubi = (b >> 1) / G;
        woff[j] = (uint32_t)((((u0 / 16 + ubi) * G + g) * nkg + kgi) * 1024 + lane * 16);
    }
}

// One tile: rows [TM*(tile / nut), +TM) x units [TU*(tile % nut), +TU) of the
// batch, all gates.  st0 / st1: the kernel's two LDS stages.
template <int KIND, typename T, int VB>
__device__ __forceinline__ void big_tile(const BatchArgs& a, int tile, char* st0, char* st1) {
    using KT = Kind<KIND>;
    constexpr uint32_t ES = sizeof(T);
    constexpr int BK = big_bk<T>(), PV = 16 / (int)sizeof(T);   // k values per chunk, per 16-byte piece
    constexpr int G = KT::G, NFX = KT::NFIX;
    constexpr int RB = big_rb(G, VB), CU = big_cu(VB);
    constexpr int TM = 32 * RB, TU = 32 * CU;
    constexpr int NSEG = (KT::X ? 1 : 0) + NFX;
    constexpr int NBW = CU * G;                      // weight blocks per wave per chunk
    constexpr int SB = big_stage_bytes<G, RB, CU>();
    constexpr int A_BYTES = TM * 128;
    static_assert(!KT::RAG, "ragged kinds use the small tile");
    static_assert(NSEG >= 1, "a cell has at least one operand segment");

    const int nut = a.Hu / TU;
    const int row0 = (tile / nut) * TM, u0 = (tile % nut) * TU;
    const int nrows = min(TM, a.m - row0);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = wave >> 1, wc = wave & 1;
    const int E = a.E, Ep = a.Ep, H = a.H, Hk = a.Hk;
    const int nkg = a.K / Elem<T>::KG;
    const int nch = a.K / BK;        // segments are whole chunks (checked by the host)

    // ---- operand copies: buffer -> LDS, 32-bit byte offsets; a masked piece
    // uses an offset past the buffer and arrives as zero, so the copies carry
    // no branches.  Buffers stay below 2^31 bytes (checked by the host); the
    // offsets are unsigned so that OOB plus a column stays out of range ----
    constexpr uint32_t OOB = 0x80000000u;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.xmat, KT::X ? (uint32_t)a.n_xrows * (uint32_t)E * ES : 0u);
    const __amdgpu_buffer_rsrc_t rh = make_rsrc(a.arena_h, (uint32_t)a.n_slots * (uint32_t)H * ES);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(a.W, (uint32_t)(a.Hu / 16) * G * nkg * 1024u);

    // A copies: wave w's j-th copy fills rows (4 j + w) * 8 .. + 8 of the stage;
    // lane l writes slot l & 7 of row (4 j + w) * 8 + l / 8, which holds piece
    // q = (l & 7) ^ (l / 8) of that row.
    const int q = (lane & 7) ^ (lane >> 3);
    uint32_t soff[NSEG][RB];   // byte offset of each segment's source row (OOB: zero)
    uint32_t woff[NBW];
    big_offsets<KIND, T, VB, NSEG, RB, NBW>(a, tile, wave, lane, soff, woff);

    v4f acc[CU][G][RB];
#pragma unroll
    for (int cu = 0; cu < CU; ++cu)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) acc[cu][g][rb] = v4f{0.f, 0.f, 0.f, 0.f};

    // ---- double-buffered chunk pipeline: the copies of chunk c+1 run while
    // the matrix cores work on chunk c; the barrier waits for them.  The
    // chunk's segment is tracked incrementally (uniform scalars).  Even
    // chunks live in st0, odd chunks in st1 ----
    int sg = 0, scol = 0, slim = KT::X ? E : H, send = KT::X ? Ep : Hk;
    auto next_seg = [&]() {
        scol += BK;
        if (scol >= send) { ++sg; scol = 0; slim = H; send = Hk; }
    };
    big_copy<T, RB, NSEG, NBW, KT::X>(soff, woff, rx, rh, rw, 0, sg, scol + q * PV, slim, st0, st0 + A_BYTES, wave);
    __syncthreads();
    int c = 0;
    for (; c + 1 < nch; c += 2) {
        next_seg();
        big_copy<T, RB, NSEG, NBW, KT::X>(soff, woff, rx, rh, rw, c + 1, sg, scol + q * PV, slim, st1,
                                         st1 + A_BYTES, wave);
        big_compute<T, RB, CU, G>(acc, st0, reinterpret_cast<const uint4*>(st0 + A_BYTES), wr, wc, lane);
        __syncthreads();
        if (c + 2 < nch) {
            next_seg();
            big_copy<T, RB, NSEG, NBW, KT::X>(soff, woff, rx, rh, rw, c + 2, sg, scol + q * PV, slim, st0,
                                             st0 + A_BYTES, wave);
        }
        big_compute<T, RB, CU, G>(acc, st1, reinterpret_cast<const uint4*>(st1 + A_BYTES), wr, wc, lane);
        __syncthreads();
    }
    if (c < nch) big_compute<T, RB, CU, G>(acc, st0, reinterpret_cast<const uint4*>(st0 + A_BYTES), wr, wc, lane);
    __syncthreads();   // the stages are free for the epilogue's operands

    // ---- epilogue operands, copied into the stage buffers: rows of 64 fp32
    // values from the tile's first unit (its TU units, and for the narrow
    // classes 32 more that go unused; past the arena they read as zero), the
    // first half of each list in st0 and the
    // second in st1.  Cell kinds: the positional children's cell states.  The
    // forget GEMM: the children's own cell states.  The parent GEMM: the sums
    // of the children's products sigma(f_k) c_k (one row per parent) ----
    constexpr int HALF = TM / 2;
    constexpr int NCR = big_ncr<KIND>();
    // the epilogue's own loads (bias, result rows), issued with the copies of
    // the children's rows below
    float bz[CU][G];   // bias of this lane's units (the packed bias is zero-padded to Hu)
#pragma unroll
    for (int cu = 0; cu < CU; ++cu)
#pragma unroll
        for (int g = 0; g < G; ++g) bz[cu][g] = a.bias[g * a.Hu + u0 + (wc * CU + cu) * 16 + (lane & 15)];
    int rres[RB][4];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = min(wr * 16 * RB + rb * 16 + (lane >> 4) * 4 + i, nrows - 1);
            rres[rb][i] = KIND == K_CS_FORGET ? row0 + r : seg_row(a.res, row0 + r);
        }
    static_assert(NCR * HALF * 256 <= SB, "epilogue rows fit the stages");
    const __amdgpu_buffer_rsrc_t rc = KIND == K_CS_PARENT
                                          ? make_rsrc(a.fc, (uint32_t)a.m * (uint32_t)H * 4u)
                                          : make_rsrc(a.arena_c, (uint32_t)a.n_slots * (uint32_t)H * 4u);
    auto crow_ptr = [&](int p, int r) -> const float* {
        const char* base = r < HALF ? st0 : st1;
        return reinterpret_cast<const float*>(base + (p * HALF + (r < HALF ? r : r - HALF)) * 256);
    };
    if constexpr (NCR > 0) {
#pragma unroll
        for (int p = 0; p < NCR; ++p)
#pragma unroll
            for (int j = 0; j < TM / 16; ++j) {
                const int r0 = (4 * j + wave) * 4;              // first of the copy's 4 rows (uniform)
                const int r = r0 + (lane >> 4);
                int srow = -1;
                if (r < nrows) {
                    if constexpr (KIND == K_CS_FORGET) srow = seg_row(a.x, row0 + r);
                    else if constexpr (KIND == K_CS_PARENT) srow = row0 + r;
                    else srow = a.fix[p].kind == S_NONE ? -1 : seg_row(a.fix[p], row0 + r);
                }
                const uint32_t off = srow >= 0 ? ((uint32_t)srow * (uint32_t)H + (uint32_t)u0) * 4u +
                                                     (uint32_t)(lane & 15) * 16u
                                               : OOB;
                char* dst = (r0 < HALF ? st0 : st1) + (p * HALF + (r0 < HALF ? r0 : r0 - HALF)) * 256;
                dma16(rc, off, dst);
            }
        __syncthreads();
    }

    // ---- gate epilogue: every element's new c and h in registers (the
    // children's cell states are still in the stages) ----
    constexpr bool FORGET = KIND == K_CS_FORGET;
    float cv[RB][4][CU], hv[RB][4][CU];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = min(wr * 16 * RB + rb * 16 + (lane >> 4) * 4 + i, TM - 1);
#pragma unroll
            for (int cu = 0; cu < CU; ++cu) {
                const int u = (wc * CU + cu) * 16 + (lane & 15);
                float z[G], cp[NFX > 0 ? NFX : 1];
#pragma unroll
                for (int g = 0; g < G; ++g) z[g] = acc[cu][g][rb][i] + bz[cu][g];
                cp[0] = 0.f;
#pragma unroll
                for (int p = 0; p < NCR; ++p) cp[p] = crow_ptr(p, r)[u];
                if constexpr (FORGET) {
                    cv[rb][i][cu] = sigm(z[0]) * cp[0];   // sigma(f_k) c_k, row = position in the child list
                    hv[rb][i][cu] = 0.f;
                } else if constexpr (KIND == K_CS_PARENT) {
                    cell_update<K_CS_INT>(z, cp, cp[0], 0.f, 0, cv[rb][i][cu], hv[rb][i][cu]);
                } else {
                    cell_update<KIND>(z, cp, 0.f, 0.f, 0, cv[rb][i][cu], hv[rb][i][cu]);
                }
            }
            // one row at a time: keeps the unrolled epilogue's live registers small
            __builtin_amdgcn_sched_barrier(0);
        }
    if constexpr (NCR > 0) __syncthreads();   // every read of the children's cell states is done
    (void)rres;

    // ---- scatter through LDS: per row block rb, the 32 rows it covers (16 of
    // each row half) go to the stages as [32][TU] tiles (c fp32 in st0, h in
    // st1, rows padded by 16 bytes so that the 4 rows one store instruction
    // covers fall in distinct banks), then every thread writes whole 16-byte
    // pieces of those rows to their slots: each row's TU units are contiguous
    // in its slot ----
    constexpr int CS = TU + 4;                       // c tile row stride (floats)
    constexpr int HS = TU + 16 / (int)sizeof(T);     // h tile row stride (elements)
    static_assert(32 * CS * 4 <= SB && 32 * HS * (int)sizeof(T) <= SB, "an output pass fits a stage");
    float* Cs = reinterpret_cast<float*>(st0);
    T* Hs = reinterpret_cast<T*>(st1);
    T* Hout = reinterpret_cast<T*>(a.arena_h);
    constexpr int CP = TU / 4, HP = TU * (int)sizeof(T) / 16;   // 16-byte pieces of a row of c, of h
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int lr = wr * 16 + (lane >> 4) * 4 + i;   // row in the pass
#pragma unroll
            for (int cu = 0; cu < CU; ++cu) {
                const int u = (wc * CU + cu) * 16 + (lane & 15);
                Cs[lr * CS + u] = cv[rb][i][cu];
                if constexpr (!FORGET) Hs[lr * HS + u] = from_f<T>(hv[rb][i][cu]);
            }
        }
        __syncthreads();
        // pass row lr is tile row (lr / 16) * 16 * RB + rb * 16 + lr % 16
        for (int pc = tid; pc < 32 * CP; pc += 256) {
            const int lr = pc / CP, qq = pc - lr * CP;
            const int r = (lr >> 4) * 16 * RB + rb * 16 + (lr & 15);
            const int j = u0 + qq * 4;
            if (r >= nrows || j >= a.H) continue;
            const int rr = FORGET ? row0 + r : seg_row(a.res, row0 + r);
            float* dst = (FORGET ? a.fc : a.arena_c) + (size_t)rr * a.H + j;
            *reinterpret_cast<float4*>(dst) = *reinterpret_cast<const float4*>(Cs + lr * CS + qq * 4);
        }
        if constexpr (!FORGET) {
            for (int ph = tid; ph < 32 * HP; ph += 256) {
                const int lr = ph / HP, qq = ph - lr * HP;
                const int r = (lr >> 4) * 16 * RB + rb * 16 + (lr & 15);
                const int j = u0 + qq * PV;
                if (r >= nrows || j >= a.H) continue;
                const int rr = seg_row(a.res, row0 + r);
                *reinterpret_cast<uint4*>(Hout + (size_t)rr * a.H + j) =
                    *reinterpret_cast<const uint4*>(Hs + lr * HS + qq * PV);
            }
        }
        __syncthreads();   // the next pass overwrites the tiles
    }
}

// Two stages as distinct objects: the compiler can then tell that the copies
// into one stage do not alias the reads of the other and does not wait for
// the copies before the reads.
#define EDB_BIG_STAGES(KIND, VB)                                                                       \
    constexpr int SB_ = big_stage_bytes<Kind<KIND>::G, big_rb(Kind<KIND>::G, VB), big_cu(VB)>();      \
    __shared__ __align__(16) char st0[SB_];                                                         \
    __shared__ __align__(16) char st1[SB_]

// Waves per SIMD the compiler is held to: two work-groups per CU where the
// accumulators (4 CU G RB registers) leave room for them, else one.
template <int KIND, int VB>
__host__ __device__ constexpr int big_waves_per_simd() {
    return 4 * big_cu(VB) * Kind<KIND>::G * big_rb(Kind<KIND>::G, VB) <= 96 ? 2 : 1;
}

// One work-group per tile, in XCD-aware order: work-groups are dispatched
// round-robin over the 8 XCDs and XCD x owns the contiguous tile range
// [x per, (x + 1) per), unit tiles fastest.  The grid is a multiple of 8.
template <int KIND, typename T, int VB>
__global__ __launch_bounds__(256, (big_waves_per_simd<KIND, VB>())) void big_kernel(BatchArgs a) {
    EDB_BIG_STAGES(KIND, VB);
    constexpr int TM = 32 * big_rb(Kind<KIND>::G, VB), TU = 32 * big_cu(VB);
    const int nut = a.Hu / TU;
    const int ntile = ((a.m + TM - 1) / TM) * nut;
    const int per = (ntile + 7) / 8;
    const int tile = (int)(blockIdx.x & 7) * per + (int)(blockIdx.x >> 3);
    clear_zero_rows<T>(a);
    if (tile >= ntile) return;
    big_tile<KIND, T, VB>(a, tile, st0, st1);
}

// Per parent of a child-sum batch, after the forget GEMM: the child sum of h,
// hsum[r] = bf16(sum of the children's h rows, fp32, in child order) (the
// rounding of the small tile's child-sum staging), and the sum of the
// children's products, racc[r] = sum_k sigma(f_k) c_k in child order.  One
// thread per 8 units of a row.
__global__ __launch_bounds__(256) void child_reduce_kernel(BatchArgs a, __bf16* __restrict__ hsum,
                                                           float* __restrict__ racc) {
    using T = __bf16;
    const int nv = a.H / 8;
    const int it = blockIdx.x * 256 + threadIdx.x;
    if (it >= a.m * nv) return;
    const int r = it / nv, c = it - r * nv;
    const T* h = reinterpret_cast<const T*>(a.arena_h);
    const int e0 = a.rag_ptr[r], e1 = a.rag_ptr[r + 1];
    float acc[8], sf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = sf[i] = 0.f;
    int e = e0;
    for (; e + 4 <= e1; e += 4) {
        uint4 raw[4];
        float4 f[4][2];
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            raw[n] = *reinterpret_cast<const uint4*>(h + (size_t)seg_row(a.rag, e + n) * a.H + c * 8);
            f[n][0] = *reinterpret_cast<const float4*>(a.fc + (size_t)(e + n) * a.H + c * 8);
            f[n][1] = *reinterpret_cast<const float4*>(a.fc + (size_t)(e + n) * a.H + c * 8 + 4);
        }
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            const T* pv = reinterpret_cast<const T*>(&raw[n]);
            const float* pf = reinterpret_cast<const float*>(&f[n][0]);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                acc[i] += to_f(pv[i]);
                sf[i] += pf[i];
            }
        }
    }
    for (; e < e1; ++e) {
        const uint4 raw = *reinterpret_cast<const uint4*>(h + (size_t)seg_row(a.rag, e) * a.H + c * 8);
        float4 f[2];
        f[0] = *reinterpret_cast<const float4*>(a.fc + (size_t)e * a.H + c * 8);
        f[1] = *reinterpret_cast<const float4*>(a.fc + (size_t)e * a.H + c * 8 + 4);
        const T* pv = reinterpret_cast<const T*>(&raw);
        const float* pf = reinterpret_cast<const float*>(&f[0]);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            acc[i] += to_f(pv[i]);
            sf[i] += pf[i];
        }
    }
    uint4 o;
    T* po = reinterpret_cast<T*>(&o);
#pragma unroll
    for (int i = 0; i < 8; ++i) po[i] = from_f<T>(acc[i]);
    *reinterpret_cast<uint4*>(hsum + (size_t)r * a.H + c * 8) = o;
    *reinterpret_cast<float4*>(racc + (size_t)r * a.H + c * 8) = make_float4(sf[0], sf[1], sf[2], sf[3]);
    *reinterpret_cast<float4*>(racc + (size_t)r * a.H + c * 8 + 4) = make_float4(sf[4], sf[5], sf[6], sf[7]);
}

}  // namespace edbk
