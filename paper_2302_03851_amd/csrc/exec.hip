// Device executor: weight packing, per-batch launch records, HIP graph
// capture and replay of the whole batch sequence.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <atomic>
#include <map>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "big_tile.h"
#include "ws_tile.h"
#include "cell_kernels.h"
#include "diag_kernels.h"
#include "mv_kernels.h"
#include "edb_internal.h"

using edb::fail;
using namespace edbk;

namespace {

constexpr int NUM_SMALL = 8;
constexpr int NUM_LARGE = 3;        // large size classes 0-2 (variants 8-10)
constexpr int NUM_STREAM = 4;
constexpr int FIRST_STREAM = NUM_SMALL + NUM_LARGE;
constexpr int FIRST_NARROW = FIRST_STREAM + NUM_STREAM;   // large size classes 3-4 (variants 15-16)
constexpr int WS_VARIANT = FIRST_NARROW + NUM_BIG_CLASSES - NUM_LARGE;   // the weight-stationary tile
constexpr int NUM_VARIANTS = WS_VARIANT + 1;
// small (staged) and streamed tile variants: rows per work-group 16*RT, units
// per work-group 16*WU, WK waves splitting the reduction (threads per
// work-group 64*WU*WK); the large variants have no entry here
constexpr int VAR_RT[NUM_VARIANTS] = {2, 1, 1, 1, 1, 1, 2, 2, 0, 0, 0, 1, 2, 1, 1, 0, 0, 0};
constexpr int VAR_WU[NUM_VARIANTS] = {4, 4, 2, 1, 1, 1, 1, 2, 0, 0, 0, 1, 1, 1, 1, 0, 0, 0};
constexpr int VAR_WK[NUM_VARIANTS] = {1, 1, 2, 4, 8, 16, 4, 2, 0, 0, 0, 4, 4, 8, 16, 0, 0, 0};
// large tile variants 8-10 and 15-16 = size classes 0-4: 32*big_rb(G, vb) rows x
// 32*big_cu(vb) units, 256 threads (bf16 and fp32; chunks of 128 bytes of k)
bool is_large(int v) { return (v >= NUM_SMALL && v < FIRST_STREAM) || (v >= FIRST_NARROW && v < WS_VARIANT); }
bool is_ws(int v) { return v == WS_VARIANT; }
int large_class(int v) { return v < FIRST_STREAM ? v - NUM_SMALL : v - FIRST_NARROW + NUM_LARGE; }
int large_variant(int vb) { return vb < NUM_LARGE ? NUM_SMALL + vb : FIRST_NARROW + vb - NUM_LARGE; }
// streamed tile variants FIRST_STREAM..: 16*RT rows x 16 units, WK waves
bool is_stream(int v) { return v >= FIRST_STREAM && v < FIRST_NARROW; }
bool is_small(int v) { return v >= 0 && v < NUM_SMALL; }
// the staged variant with the same rows and reduction split as streamed variant v
constexpr int STAGED_OF[NUM_STREAM] = {3, 6, 4, 5};

struct KindInfo {
    int G, nfix;
    bool x, rag;
};

KindInfo kind_info(int kind) {
    switch (kind) {
        case EDB_CELL_LSTM_CHAIN: return {4, 1, true, false};
        case EDB_CELL_NARY_LEAF: return {3, 0, true, false};
        case EDB_CELL_NARY_INTERNAL: return {5, 2, false, false};
        case EDB_CELL_GRID: return {5, 2, true, false};
        case EDB_CELL_CS_LEAF: return {3, 0, true, false};
        case EDB_CELL_CS_INTERNAL: return {3, 0, false, true};
        case EDB_CELL_LAT_CHAR: return {5, 1, true, true};
        case EDB_CELL_LAT_WORD: return {3, 1, true, false};
        case EDB_CELL_GRU_LEAF: return {2, 0, true, false};
        case EDB_CELL_GRU_INTERNAL: return {5, 2, false, false};
        case EDB_CELL_LINEAR: return {1, 0, true, false};
        case EDB_CELL_MV_MAT: return {1, 2, false, false};
        // operand lists: the two children's vectors, then 2H matrix columns
        case EDB_CELL_MV_VEC: return {1, 2, false, true};
        case EDB_CELL_LGRU_EDGE: return {4, 1, true, false};
        case EDB_CELL_POOL_MEAN: return {1, 0, false, true};
        default: return {0, 0, false, false};
    }
}

int round_up(int v, int m) { return (v + m - 1) / m * m; }

// Derived dimensions of a cell type's packed layout.
struct Dims {
    int G, KG, esz, E, Ep, H, Hk, Hu, K;
    bool x, rag;
    int64_t off_W, off_b, off_Wr, off_br, bytes;
};

edb_status cell_dims(const edb_cell* c, Dims& d) {
    if (!c) return fail(EDB_ERR_INVALID, "cell is NULL");
    KindInfo ki = kind_info(c->kind);
    if (ki.G == 0) return fail(EDB_ERR_INVALID, "unknown cell kind " + std::to_string(c->kind));
    // an MV-RNN vector batch's GEMM reads the rows [B a, A b] (2H wide) as its
    // x operand; its operand lists feed mv_matvec_kernel
    const bool mv_vec = c->kind == EDB_CELL_MV_VEC;
    if (mv_vec) ki = KindInfo{1, 0, true, false};
    // a pooling node's GEMM reads the sum of its ragged children (no ragged weights)
    const bool pool = c->kind == EDB_CELL_POOL_MEAN;
    if (pool) ki = KindInfo{1, 0, false, false};
    if (c->dtype != EDB_F32 && c->dtype != EDB_BF16) return fail(EDB_ERR_INVALID, "unknown cell dtype");
    if ((c->kind == EDB_CELL_LINEAR || c->kind == EDB_CELL_MV_MAT || mv_vec) && c->dtype != EDB_F32)
        return fail(EDB_ERR_UNSUPPORTED, "the MV-RNN cells (LINEAR, MV_MAT, MV_VEC) run in fp32 only");
    if ((c->kind == EDB_CELL_LGRU_EDGE || pool) && c->dtype != EDB_F32)
        return fail(EDB_ERR_UNSUPPORTED, "the lattice GRU cells (LGRU_EDGE, POOL_MEAN) run in fp32 only");
    if (c->hidden <= 0) return fail(EDB_ERR_INVALID, "hidden must be positive");
    if (ki.x && c->in_dim <= 0) return fail(EDB_ERR_INVALID, "in_dim must be positive for this cell kind");
    if (c->kind == EDB_CELL_NARY_INTERNAL && c->n_children != 2)
        return fail(EDB_ERR_UNSUPPORTED, "NARY_INTERNAL supports n_children == 2 only");
    d.G = ki.G;
    d.x = ki.x;
    d.rag = ki.rag;
    d.KG = c->dtype == EDB_F32 ? 16 : 32;
    d.esz = c->dtype == EDB_F32 ? 4 : 2;
    const int vec = 16 / d.esz;
    d.H = c->hidden;
    d.E = mv_vec ? 2 * c->hidden : ki.x ? c->in_dim : 0;
    if (d.H % vec != 0 || d.E % vec != 0)
        return fail(EDB_ERR_UNSUPPORTED, "hidden and in_dim must be multiples of " + std::to_string(vec) +
                                             " (16-byte rows)");
    if (d.H > 4096 || d.E > 4096) return fail(EDB_ERR_UNSUPPORTED, "hidden / in_dim above 4096");
    d.Hk = round_up(d.H, d.KG);
    d.Ep = ki.x ? round_up(d.E, d.KG) : 0;
    d.Hu = round_up(d.H, 64);
    if (c->kind == EDB_CELL_CS_INTERNAL || pool) d.K = d.Hk;
    else d.K = d.Ep + ki.nfix * d.Hk;
    const int64_t wmain = (int64_t)(d.Hu / 16) * d.G * (d.K / d.KG) * 64 * 16;
    const int64_t bmain = (int64_t)d.G * d.Hu * 4;
    const int64_t wr = ki.rag ? (int64_t)(d.Hu / 16) * (d.Hk / d.KG) * 64 * 16 : 0;
    const int64_t brr = ki.rag ? (int64_t)d.Hu * 4 : 0;
    auto al = [](int64_t v) { return (v + 255) / 256 * 256; };
    d.off_W = 0;
    d.off_b = al(wmain);
    d.off_Wr = d.off_b + al(bmain);
    d.off_br = d.off_Wr + al(wr);
    d.bytes = d.off_br + al(brr);
    return EDB_OK;
}

uint16_t bf16_rne(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Logical row of main-GEMM K position k (padded layout), or -1 for padding.
int main_row(int kind, const Dims& d, int k) {
    int seg_start = 0, logical_start = 0;
    if (d.x) {
        if (k < d.Ep) return k < d.E ? k : -1;
        seg_start = d.Ep;
        logical_start = d.E;
    }
    const int s = (k - seg_start) / d.Hk, o = (k - seg_start) % d.Hk;
    (void)kind;
    return o < d.H ? logical_start + s * d.H + o : -1;
}

// Pack one GEMM operand [K x (G x H)] into the lane layout of cell_kernels.h.
void pack_gemm(std::vector<uint8_t>& out, int64_t off, const Dims& d, int G, int K,
               const std::function<float(int k, int g, int j)>& val) {
    const int nkg = K / d.KG, per = d.KG / 4;
    for (int ub = 0; ub < d.Hu / 16; ++ub)
        for (int g = 0; g < G; ++g)
            for (int kg = 0; kg < nkg; ++kg)
                for (int l = 0; l < 64; ++l)
                    for (int i = 0; i < per; ++i) {
                        const int k = kg * d.KG + (l / 16) * per + i;
                        const int j = ub * 16 + (l % 16);
                        const float v = j < d.H ? val(k, g, j) : 0.f;
                        const int64_t e = ((((int64_t)ub * G + g) * nkg + kg) * 64 + l) * per + i;
                        if (d.esz == 4) std::memcpy(out.data() + off + e * 4, &v, 4);
                        else {
                            uint16_t b = bf16_rne(v);
                            std::memcpy(out.data() + off + e * 2, &b, 2);
                        }
                    }
}

}  // namespace

extern "C" edb_status edb_packed_weight_bytes(const edb_cell* cell, int64_t* bytes) {
    if (!bytes) return fail(EDB_ERR_INVALID, "edb_packed_weight_bytes: bytes is NULL");
    Dims d;
    edb_status st = cell_dims(cell, d);
    if (st != EDB_OK) return st;
    *bytes = d.bytes;
    return EDB_OK;
}

extern "C" edb_status edb_pack_weights(const edb_cell* cell, const float* const* lg, void* packed_dev,
                                       void* stream) {
    Dims d;
    edb_status st = cell_dims(cell, d);
    if (st != EDB_OK) return st;
    if (!lg || !packed_dev) return fail(EDB_ERR_INVALID, "edb_pack_weights: NULL argument");
    const int nmat = cell->kind == EDB_CELL_CS_INTERNAL ? 4 : cell->kind == EDB_CELL_LAT_CHAR ? 5 : 2;
    for (int i = 0; i < nmat; ++i)
        if (!lg[i]) return fail(EDB_ERR_INVALID, "edb_pack_weights: NULL logical matrix");
    std::vector<uint8_t> buf;
    try {
        buf.assign((size_t)d.bytes, 0);
    } catch (const std::bad_alloc&) {
        return fail(EDB_ERR_OOM, "edb_pack_weights: out of host memory");
    }
    const int kind = cell->kind, H = d.H, G = d.G;
    const float *W = lg[0], *b = nullptr, *Wr = nullptr, *br = nullptr, *Wlx = nullptr;
    int ncol = 0;  // logical columns of W
    switch (kind) {
        case EDB_CELL_CS_INTERNAL: ncol = 3 * H; Wr = lg[1]; b = lg[2]; br = lg[3]; break;
        case EDB_CELL_LAT_CHAR: ncol = 4 * H; Wlx = lg[1]; Wr = lg[2]; b = lg[3]; br = lg[4]; break;
        default: ncol = G * H; b = lg[1]; break;
    }
    pack_gemm(buf, d.off_W, d, G, d.K, [&](int k, int g, int j) -> float {
        const int row = main_row(kind, d, k);
        if (row < 0) return 0.f;
        if (kind == EDB_CELL_LAT_CHAR && g == 4) return row < d.E ? Wlx[(int64_t)row * H + j] : 0.f;
        // TreeGRU candidates: n_0 reads only child 0's rows, n_1 only child 1's
        if (kind == EDB_CELL_GRU_INTERNAL && ((g == 3 && row >= H) || (g == 4 && row < H))) return 0.f;
        // lattice GRU edge: n_x reads only x's rows, n_h only the source state's
        if (kind == EDB_CELL_LGRU_EDGE && ((g == 2 && row >= d.E) || (g == 3 && row < d.E))) return 0.f;
        return W[(int64_t)row * ncol + g * H + j];
    });
    float* bias = reinterpret_cast<float*>(buf.data() + d.off_b);
    for (int g = 0; g < G; ++g)
        for (int j = 0; j < H; ++j)
            bias[g * d.Hu + j] = (kind == EDB_CELL_LAT_CHAR && g == 4) ? 0.f : b[g * H + j];
    if (d.rag) {
        pack_gemm(buf, d.off_Wr, d, 1, d.Hk, [&](int k, int, int j) -> float {
            return k < H ? Wr[(int64_t)k * H + j] : 0.f;
        });
        float* brp = reinterpret_cast<float*>(buf.data() + d.off_br);
        for (int j = 0; j < H; ++j) brp[j] = br[j];
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(packed_dev, buf.data(), (size_t)d.bytes, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_pack_weights: ") + hipGetErrorString(e));
    return EDB_OK;
}

// ---------------------------------------------------------------------------
// kernel dispatch

namespace {

using AttrFn = hipError_t (*)(int lds);

template <int KIND, typename T, int RT, int WU, int WK>
hipError_t attr_cell(int lds) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&cell_kernel<KIND, T, RT, WU, WK>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}
template <int KIND, typename T, int RT, int WU, int WK>
int lds_cell(int K, int Hk) { return lds_bytes<KIND, T, RT, WU, WK>(K, Hk); }

// A kernel variant: its LDS attribute setter, its LDS size and the kernel
// (null where the variant does not serve the kind).
struct Entry {
    AttrFn attr;
    int (*lds)(int K, int Hk);   // LDS bytes for reduction length K and ragged row width Hk
    const void* fn;   // the kernel (launches, graph nodes and occupancy queries)
};

template <int KIND, typename T, int RT, int WU, int WK>
Entry entry() {
    return {attr_cell<KIND, T, RT, WU, WK>, lds_cell<KIND, T, RT, WU, WK>,
            reinterpret_cast<const void*>(&cell_kernel<KIND, T, RT, WU, WK>)};
}

// the weight-stationary tile (bf16 leaf kinds): dynamic LDS for the weights
template <int KIND>
hipError_t attr_ws(int lds) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&ws_kernel<KIND>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}
template <int KIND>
int lds_ws(int K, int) { return ws_lds_bytes(Kind<KIND>::G, K); }

template <int KIND, typename T>
Entry ws_entry() {
    if constexpr (ws_kind<KIND>() && sizeof(T) == 2)
        return {attr_ws<KIND>, lds_ws<KIND>, reinterpret_cast<const void*>(&ws_kernel<KIND>)};
    else return {nullptr, nullptr, nullptr};
}

template <int KIND, int VB>
hipError_t attr_big(int) { return hipSuccess; }
template <int KIND, int VB>
int lds_big(int, int) { return big_lds_bytes<KIND, VB>(); }

template <int KIND, typename T, int VB>
Entry big_entry() {
    if constexpr (!Kind<KIND>::RAG && !sums_children<KIND>())
        return {attr_big<KIND, VB>, lds_big<KIND, VB>,
                reinterpret_cast<const void*>(&big_kernel<KIND, T, VB>)};
    else return {nullptr, nullptr, nullptr};
}

template <int KIND, typename T, int RT, int WK>
hipError_t attr_stream(int lds) {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&stream_kernel<KIND, T, RT, WK>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, lds);
}
template <int KIND, typename T, int RT, int WK>
int lds_stream(int, int) { return stream_lds_bytes<KIND, T, RT, WK>(); }

// the streamed tile serves the kinds without a ragged phase
template <int KIND, typename T, int RT, int WK>
Entry stream_entry() {
    if constexpr (Kind<KIND>::RAG || sums_children<KIND>()) return {nullptr, nullptr, nullptr};
    else
        return {attr_stream<KIND, T, RT, WK>, lds_stream<KIND, T, RT, WK>,
                reinterpret_cast<const void*>(&stream_kernel<KIND, T, RT, WK>)};
}

// Rows and units per work-group of large size class vb for G gates.
int large_tm(int G, int vb) { return 32 * big_rb(G, vb); }
int large_tu(int vb) { return 32 * big_cu(vb); }

template <int KIND, typename T>
void fill_kind(Entry* e) {
    e[0] = entry<KIND, T, 2, 4, 1>();
    e[1] = entry<KIND, T, 1, 4, 1>();
    e[2] = entry<KIND, T, 1, 2, 2>();
    e[3] = entry<KIND, T, 1, 1, 4>();
    e[4] = entry<KIND, T, 1, 1, 8>();
    e[5] = entry<KIND, T, 1, 1, 16>();
    e[6] = entry<KIND, T, 2, 1, 4>();
    e[7] = entry<KIND, T, 2, 2, 2>();
    e[8] = big_entry<KIND, T, 0>();
    e[9] = big_entry<KIND, T, 1>();
    e[10] = big_entry<KIND, T, 2>();
    e[11] = stream_entry<KIND, T, 1, 4>();
    e[12] = stream_entry<KIND, T, 2, 4>();
    e[13] = stream_entry<KIND, T, 1, 8>();
    e[14] = stream_entry<KIND, T, 1, 16>();
    e[15] = big_entry<KIND, T, 3>();
    e[16] = big_entry<KIND, T, 4>();
    e[WS_VARIANT] = ws_entry<KIND, T>();
}

// The internal kinds of a child-sum batch on the large tile have large bf16 variants only.
template <int KIND>
void fill_internal(Entry (&e)[2][NUM_VARIANTS]) {
    for (int d = 0; d < 2; ++d)
        for (int v = 0; v < NUM_VARIANTS; ++v) e[d][v] = {nullptr, nullptr, nullptr};
    e[1][8] = big_entry<KIND, __bf16, 0>();
    e[1][9] = big_entry<KIND, __bf16, 1>();
    e[1][10] = big_entry<KIND, __bf16, 2>();
    e[1][15] = big_entry<KIND, __bf16, 3>();
    e[1][16] = big_entry<KIND, __bf16, 4>();
}

constexpr int kWsMinRows = 8192;   // batches the weight-stationary tile takes (at least)
constexpr int NUM_KERNEL_KINDS = 17;   // the 15 cell kinds, then K_CS_FORGET, K_CS_PARENT

struct Table {
    Entry e[NUM_KERNEL_KINDS][2][NUM_VARIANTS];
    Table() {
        fill_kind<K_CHAIN, float>(e[0][0]);        fill_kind<K_CHAIN, __bf16>(e[0][1]);
        fill_kind<K_NARY_LEAF, float>(e[1][0]);    fill_kind<K_NARY_LEAF, __bf16>(e[1][1]);
        fill_kind<K_NARY_INT, float>(e[2][0]);     fill_kind<K_NARY_INT, __bf16>(e[2][1]);
        fill_kind<K_GRID, float>(e[3][0]);         fill_kind<K_GRID, __bf16>(e[3][1]);
        fill_kind<K_CS_LEAF, float>(e[4][0]);      fill_kind<K_CS_LEAF, __bf16>(e[4][1]);
        fill_kind<K_CS_INT, float>(e[5][0]);       fill_kind<K_CS_INT, __bf16>(e[5][1]);
        fill_kind<K_LAT_CHAR, float>(e[6][0]);     fill_kind<K_LAT_CHAR, __bf16>(e[6][1]);
        fill_kind<K_LAT_WORD, float>(e[7][0]);     fill_kind<K_LAT_WORD, __bf16>(e[7][1]);
        fill_kind<K_GRU_LEAF, float>(e[8][0]);     fill_kind<K_GRU_LEAF, __bf16>(e[8][1]);
        fill_kind<K_GRU_INT, float>(e[9][0]);      fill_kind<K_GRU_INT, __bf16>(e[9][1]);
        // the MV-RNN kinds run in fp32 only (cell_dims rejects bf16 for them)
        fill_kind<K_LINEAR, float>(e[10][0]);
        fill_kind<K_MV_MAT, float>(e[11][0]);
        fill_kind<K_MV_VEC, float>(e[12][0]);
        // the lattice GRU kinds run in fp32 only; the pooling node on the staged tile only
        fill_kind<K_LGRU_EDGE, float>(e[13][0]);
        fill_kind<K_POOL_MEAN, float>(e[14][0]);
        fill_internal<K_CS_FORGET>(e[K_CS_FORGET]);
        fill_internal<K_CS_PARENT>(e[K_CS_PARENT]);
    }
};

const Table& table() {
    static Table t;
    return t;
}

// One kernel launch of the forward pass.
struct Launch {
    edb_launch_info info;
    int type;      // cell type (batches)
    int kk = 0;    // kernel kind (the cell kind, or K_CS_FORGET / K_CS_PARENT)
    BatchArgs args;  // pointer fields to data buffers are filled at execute time
    // offsets into the device int buffer (-1 = none)
    int64_t off_x, off_f0, off_f1, off_rag, off_rptr, off_res;
    int64_t off_zrows = -1;   // the first batch clears the zero and pad rows listed here
    int x_base;
    int lds;
    // dataflow launch (info.variant == FLOW_VARIANT): offsets into the int buffer
    bool flow = false;
    int64_t f_desc, f_tiles, f_rtdeps, f_deps, f_ticket, f_error, f_done;
    int f_ntiles, f_need;
};

constexpr int FLOW_VARIANT = 100;

template <typename T>
int flow_lds(const std::vector<int>& kinds_k) {
    // LDS of the largest tile body among (kind, K) pairs of the run (a ragged
    // row is at most K wide: K bounds Hk)
    int best = 0;
    for (size_t i = 0; i + 1 < kinds_k.size(); i += 2) {
        const int kind = kinds_k[i], K = kinds_k[i + 1];
        int l = 0;
        switch (kind) {
            case K_CHAIN: l = lds_bytes<K_CHAIN, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_NARY_LEAF: l = lds_bytes<K_NARY_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_NARY_INT: l = lds_bytes<K_NARY_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_GRID: l = lds_bytes<K_GRID, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_CS_LEAF: l = lds_bytes<K_CS_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_CS_INT: l = lds_bytes<K_CS_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_LAT_CHAR: l = lds_bytes<K_LAT_CHAR, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_GRU_LEAF: l = lds_bytes<K_GRU_LEAF, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            case K_GRU_INT: l = lds_bytes<K_GRU_INT, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
            default: l = lds_bytes<K_LAT_WORD, T, FLOW_RT, FLOW_WU, FLOW_WK>(K, K); break;
        }
        best = std::max(best, l);
    }
    return (best + 15) / 16 * 16;
}

// Estimated microseconds of one batch under a small (staged) or streamed tile
// variant v, occ work-groups of it resident per CU.  The work-groups run in
// rounds of n_cu * occ; each round costs a latency term plus, for the busiest
// CU's c work-groups, their matrix-core time per SIMD, the bytes they load
// (operand rows and weights) and, for the staged tile, the bytes they stage,
// and the bytes beyond 100 KB per CU (L2 bandwidth saturating); the staged
// tile adds its split-K reduction and the chunks of the ragged phase; the
// whole batch adds a term in its total loaded bytes.  The coefficients of
// each family are a non-negative least-squares fit (relative error) to
// per-launch times of every variant on every batch of the five workloads on
// MI355X (2636 launches; median error 4.4% staged, 3.5% streamed).
double variant_cost(int v, int m, const Dims& d, int dtype, int64_t nrag, int occ, int n_cu) {
    static constexpr double kStaged[11] = {0, 3.7873, 1.5822, 0, 0.0015529, 1.1881, 2.8009, 0, 7.3157, 0, 0.023189};
    static constexpr double kStream[11] = {1.4473, 1.8894, 0.88904, 0, 0, 0.50528, 0, 0, 0, 0.0068505, 0.021677};
    const double* k = is_stream(v) ? kStream : kStaged;
    const int RT = VAR_RT[v], WU = VAR_WU[v], WK = VAR_WK[v], W = WU * WK;
    const int TM = 16 * RT, TU = 16 * WU;
    const int64_t tiles = (int64_t)((m + TM - 1) / TM) * (d.Hu / TU);
    occ = std::max(occ, 1);
    const int64_t cap = (int64_t)n_cu * occ;
    const int64_t full = tiles / cap, rem = tiles % cap;
    const int nkg = d.K / d.KG;
    const double kpw = std::ceil((double)nkg / WK);
    const double cyc = dtype == EDB_F32 ? 128.0 : 16.0;   // matrix-core cycles per (k-group, gate, row block)
    const double mf = std::max(1, W / 4) * kpw * d.G * RT * cyc / 2400.0;          // us per SIMD per work-group
    const double ld = ((double)TM * d.K + (double)TU * d.G * d.K) * d.esz / 1024.0;  // KB loaded per work-group
    const double st = is_stream(v) ? 0.0 : (double)TM * d.K * d.esz / 1024.0;      // KB staged per work-group
    double chunks = 0, rkpw = 0, RTR = RT;
    if (d.rag && m > 0) {
        RTR = std::max(RT, 4);
        chunks = std::ceil((double)nrag / m * TM / (16 * RTR));
        rkpw = std::ceil((double)(d.Hk / d.KG) / WK);
    }
    const double per_round_fixed = k[1] + k[5] * WK * RT * d.G / 64.0 + k[6] * chunks +
                                   k[7] * chunks * rkpw * RTR * (dtype == EDB_F32 ? 8.0 : 1.0) / 64.0 +
                                   k[8] * chunks * rkpw / 16.0;
    auto round_us = [&](double c) {
        return per_round_fixed + c * (k[2] * mf + k[3] * ld + k[4] * st) + k[9] * std::max(0.0, c * ld - 100.0);
    };
    double t = k[0] + (double)full * round_us(occ) + k[10] * (double)tiles * ld / 1024.0;
    if (rem) t += round_us((double)((rem + n_cu - 1) / n_cu));
    // streamed tile whose waves load their whole k-range in the ring prologue,
    // with several work-groups per CU: all request their operands at once and
    // no loads overlap the matrix cores.  The linear terms miss this; the
    // factor is the measured ratio on such batches (C2's 1,858-row leaf batch).
    const int pd = WK >= 16 ? 2 : (d.G >= 5 ? 3 : 4);
    if (is_stream(v) && kpw <= pd && tiles > n_cu) t *= 1.45;
    return t;
}

// Estimated microseconds of the large tile, size class vb, for G gates over K
// (padded) and m rows, occ work-groups resident per CU.  The busiest CU runs
// T = ceil(tiles / n_cu) tiles in R = ceil(tiles / (n_cu * occ)) rounds.  The
// estimate adds a fixed term; the bytes the whole launch copies to LDS (the
// L2s' shared bandwidth); a latency term per round and 128-byte chunk of k;
// the busiest CU's matrix-core time; its LDS-copy time at about 86 GB/s; its
// epilogue elements per gate; a term per round; and, with one tile per CU,
// that tile's copy and matrix-core time, which nothing overlaps.  A tail
// round of a few tiles costs little here: it runs once the other CUs have
// finished, with the memory system to itself.  Coefficients per size class:
// non-negative least-squares fits (relative error) to the per-launch times of
// each class forced on every batch of five workloads on MI355X (611 launches;
// median error 2.0-3.7% per class).
double large_cost(int G, int vb, int m, int K, int Hu, int dtype, int occ, int n_cu) {
    static constexpr double kc[NUM_BIG_CLASSES][8] = {
        {0.93142, 10.331, 0.68536, 0.52968, 0, 1.9054, 3.0777, 0.44844},
        {2.9115, 6.0844, 0.57178, 0.71069, 0, 1.1642, 0.075934, 0.34943},
        {2.2408, 4.8979, 0.43479, 0.4966, 0, 1.3676, 0, 0.5421},
        {2.2977, 3.7322, 0.45709, 0.70584, 0, 0.078758, 0, 0.39545},
        {1.7341, 2.5833, 0.40146, 0.77375, 0.069121, 0.939, 0, 0.39636}};
    const double* k = kc[vb];
    const int RB = big_rb(G, vb), CU = big_cu(vb), TM = 32 * RB, TU = 32 * CU;
    const bool f32 = dtype == EDB_F32;
    const int64_t tiles = (int64_t)((m + TM - 1) / TM) * (Hu / TU);
    occ = std::max(1, std::min(occ, 8));
    const double T = (double)((tiles + n_cu - 1) / n_cu);
    const double R = (double)((tiles + (int64_t)n_cu * occ - 1) / ((int64_t)n_cu * occ));
    const double nch = K / (f32 ? 32 : 64);
    const double cpy = (TM * 128.0 + 2.0 * CU * G * 2 * 1024) / 1024.0;    // KB per chunk per work-group
    const double mma = 2.0 * CU * G * RB * (f32 ? 128 : 16) / 2400.0;      // us per chunk per SIMD per work-group
    return k[0] + k[1] * (double)tiles * nch * cpy / 102400.0 + k[2] * R * nch + k[3] * T * nch * mma +
           k[4] * T * nch * cpy / 86.0 + k[5] * T * TM * TU * G / 16384.0 + k[6] * R +
           (T == 1.0 ? k[7] * nch * (cpy / 86.0 + mma) : 0.0);
}

// Estimated microseconds of child_reduce_kernel over m parents (fit as above).
double child_reduce_cost(int m) { return 3.739 + 1.0300e-3 * m; }

// Work-groups of a kernel resident on one CU (block threads, dyn_lds bytes of
// dynamic LDS, lds bytes of LDS in all): from the runtime (registers and LDS)
// when a device is bound, else from LDS and waves alone.
using OccFn = std::function<int(const Entry&, int block, int dyn_lds, int lds)>;

// Best large variant of kernel kind kk for m rows, or -1.
int best_large(int kk, int dtype, int G, int m, int K, int Hu, int n_cu, int max_lds, const OccFn& occ,
               double& est, double extra_us = 0.0) {   // dtype: EDB_F32 or EDB_BF16
    int var = -1;
    est = 1e300;
    for (int vb = 0; vb < NUM_BIG_CLASSES; ++vb) {
        const Entry& en = table().e[kk][dtype][large_variant(vb)];
        if (!en.fn) continue;
        const int lds = en.lds(K, 0);   // the large tile's LDS is static
        if (lds > max_lds) continue;
        const double c = large_cost(G, vb, m, K, Hu, dtype, occ(en, 256, 0, lds), n_cu) + extra_us;
        if (c < est) { est = c; var = large_variant(vb); }
    }
    return var;
}

}  // namespace

// Per-device state shared by all executors: the LDS limit, a non-blocking
// upload stream for descriptor copies (kept for the life of the process) and
// the largest dynamic LDS size already granted to each kernel.
struct DeviceCtx {
    int max_lds = 0;
    int n_cu = 0;
    hipStream_t upload = nullptr;    // created on the first allocating prepare
    hipStream_t release = nullptr;   // stream-ordered frees wait here, off the upload path
    void* scratch = nullptr;         // this device's address of the allocation-free entry point's array
    std::map<int, int> lds_granted;
    std::map<std::pair<const void*, int>, int> occupancy;   // (kernel, dynamic LDS) -> resident work-groups per CU
    std::vector<hipEvent_t> event_pool;      // timing events of freed EDB_PROFILE executors, for reuse
};
std::mutex g_ctx_mu;
std::map<int, DeviceCtx> g_ctx;

// The device's context (attributes only; nothing is allocated).
hipError_t device_ctx(int dev, DeviceCtx** out) {
    std::lock_guard<std::mutex> lk(g_ctx_mu);
    auto it = g_ctx.find(dev);
    if (it != g_ctx.end()) {
        *out = &it->second;
        return hipSuccess;
    }
    DeviceCtx c;
    hipError_t he = hipDeviceGetAttribute(&c.max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (he == hipSuccess) he = hipDeviceGetAttribute(&c.n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (he != hipSuccess) return he;
    *out = &(g_ctx[dev] = c);
    return hipSuccess;
}

// The device's upload and release streams, created once (the device is current).
hipError_t ctx_streams(DeviceCtx* ctx) {
    std::lock_guard<std::mutex> lk(g_ctx_mu);
    hipError_t he = hipSuccess;
    if (!ctx->upload) he = hipStreamCreateWithFlags(&ctx->upload, hipStreamNonBlocking);
    if (he == hipSuccess && !ctx->release) he = hipStreamCreateWithFlags(&ctx->release, hipStreamNonBlocking);
    return he;
}

namespace {
uint64_t next_exec_id() {
    static std::atomic<uint64_t> n{0};
    return ++n;
}
}  // namespace

struct edb_exec {
    int32_t flags = 0;
    int32_t T = 0, B = 0, dtype = 0;
    int32_t n_slots = 0, n_x = 0, E = 0, H = 0;
    int32_t x_direct_rows = 0;        // rows of the caller's x the plan addresses (max x_row + 1)
    bool x_in_place = false;          // every staged row would be the caller's row: read x in place
    int64_t hsum_rows = 0, fc_rows = 0;   // scratch rows of child-sum batches on the large tile
    void* hsum = nullptr;             // [hsum_rows][H] bf16: child sums of h
    float* racc = nullptr;            // [hsum_rows][H] fp32: per parent, sum of the children's products
    float* fc = nullptr;              // [fc_rows][H] fp32: sigma(f_k) c_k per child
    int64_t mvu_rows = 0;             // rows of MV-RNN vector batches
    void* mvu = nullptr;              // [mvu_rows][2H] of the cells' dtype: [B a, A b]
    std::vector<Dims> dims;
    std::vector<edb_cell> cells;
    std::vector<Launch> launches;     // [0] = staging, then one per batch
    int32_t n_zero = 0;
    int64_t off_xsrc = 0, off_zero = 0;
    int64_t off_counters = 0, n_counters = 0;   // dataflow counters, cleared every forward
    std::vector<int32_t> hbuf;        // host copy of the device int buffer
    void* dmem = nullptr;             // one stream-ordered allocation: dbuf | xstaged | scratch rows
    bool dmem_async = true;           // allocated with hipMallocAsync
    bool dmem_owned = true;           // false: the allocation-free entry point's array
    // byte sizes of the parts of dmem (each a multiple of 256 but the last)
    size_t d_ibytes = 0, d_xbytes = 0, d_hbytes = 0, d_rbytes = 0, d_fbytes = 0, d_mbytes = 0, d_total = 0;
    int* dbuf = nullptr;
    void* xstaged = nullptr;
    hipStream_t upload = nullptr;     // the device's upload stream
    hipStream_t release = nullptr;    // the device's stream for stream-ordered frees
    hipEvent_t ready = nullptr;       // descriptors uploaded
    hipEvent_t done = nullptr;        // last execution enqueued
    bool ran = false;
    uint64_t id = next_exec_id();       // unique per executor (graph nodes record whose calls they hold)
    std::vector<hipEvent_t> events;     // EDB_PROFILE: start and stop event of every launch
    bool profiled = false;
    int device = -1;

    DeviceCtx* ctx = nullptr;

    ~edb_exec() {
        // timing events go back to the device's pool (creating them costs
        // host time on every profiled mini-batch)
        if (ctx && !events.empty()) {
            std::lock_guard<std::mutex> lk(g_ctx_mu);
            for (hipEvent_t ev : events)
                if (ev) ctx->event_pool.push_back(ev);
        } else {
            for (hipEvent_t ev : events) (void)hipEventDestroy(ev);
        }
        if (dmem && dmem_owned) {
            // free in stream order after the upload and the last execution, on a
            // stream of its own so that later uploads do not queue behind this
            // executor's kernels
            if (dmem_async) {
                (void)hipStreamWaitEvent(release, ready, 0);
                if (ran && done) (void)hipStreamWaitEvent(release, done, 0);
                (void)hipFreeAsync(dmem, release);
            } else {
                (void)hipFree(dmem);
            }
        }
        if (ready) (void)hipEventDestroy(ready);
        if (done) (void)hipEventDestroy(done);
    }
};

namespace {

// Sizes of the parts of an executor's device memory (descriptor ints, staged
// x, child-sum scratch rows, MV-RNN vector rows) and their total.
void layout_device(edb_exec* e) {
    auto al256 = [](size_t v) { return (v + 255) / 256 * 256; };
    const size_t esz = e->dtype == EDB_F32 ? 4 : 2;
    e->d_ibytes = al256(e->hbuf.size() * sizeof(int32_t));
    e->d_xbytes = (e->n_x > 0 && !(e->flags & EDB_X_DIRECT) && !e->x_in_place)
                      ? al256((size_t)e->n_x * e->E * esz) : 0;
    e->d_hbytes = al256((size_t)e->hsum_rows * e->H * 2);
    e->d_rbytes = al256((size_t)e->hsum_rows * e->H * 4);
    e->d_fbytes = al256((size_t)e->fc_rows * e->H * 4);
    e->d_mbytes = (size_t)e->mvu_rows * 2 * e->H * esz;
    e->d_total = e->d_ibytes + e->d_xbytes + e->d_hbytes + e->d_rbytes + e->d_fbytes + e->d_mbytes;
}

// Point the executor's device buffers into `base` (d_total bytes, 256-aligned).
void bind_device(edb_exec* e, void* base_ptr) {
    uint8_t* base = reinterpret_cast<uint8_t*>(base_ptr);
    e->dmem = base_ptr;
    e->dbuf = reinterpret_cast<int*>(base);
    size_t o = e->d_ibytes;
    e->xstaged = e->d_xbytes ? base + o : nullptr;
    o += e->d_xbytes;
    e->hsum = e->d_hbytes ? base + o : nullptr;
    o += e->d_hbytes;
    e->racc = e->d_rbytes ? reinterpret_cast<float*>(base + o) : nullptr;
    o += e->d_rbytes;
    e->fc = e->d_fbytes ? reinterpret_cast<float*>(base + o) : nullptr;
    o += e->d_fbytes;
    e->mvu = e->d_mbytes ? base + o : nullptr;
}

// edb_prepare; with noalloc the executor gets no device memory, no upload and
// no events (the caller binds it to memory of its own and uploads hbuf).
edb_status prepare_impl(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                        const edb_cell* cells, int32_t flags, bool noalloc, edb_exec_t** out);

}  // namespace

extern "C" edb_status edb_prepare(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                                  const edb_cell* cells, int32_t flags, edb_exec_t** out) {
    return prepare_impl(g, s, p, cells, flags, false, out);
}

namespace {

edb_status prepare_impl(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                        const edb_cell* cells, int32_t flags, bool noalloc, edb_exec_t** out) {
    if (!out) return fail(EDB_ERR_INVALID, "edb_prepare: out is NULL");
    *out = nullptr;
    if (!g || !s || !p || !cells) return fail(EDB_ERR_INVALID, "edb_prepare: NULL argument");
    if (flags & ~(EDB_USE_GRAPH | EDB_DRYRUN | EDB_FORCE_GATHER | EDB_X_DIRECT | EDB_PROFILE | EDB_NO_FLOW |
                  EDB_NO_SPLIT_K | EDB_TILE_LARGE | EDB_NO_LARGE | EDB_FLOW_DRYRUN))
        return fail(EDB_ERR_INVALID, "edb_prepare: unknown flags");
    if ((flags & EDB_FLOW_DRYRUN) && !(flags & EDB_DRYRUN))
        return fail(EDB_ERR_INVALID, "edb_prepare: EDB_FLOW_DRYRUN needs EDB_DRYRUN (dataflow launches are switched off)");
    if ((flags & EDB_TILE_LARGE) && (flags & EDB_NO_LARGE))
        return fail(EDB_ERR_INVALID, "edb_prepare: EDB_TILE_LARGE and EDB_NO_LARGE exclude each other");
    if (s->V != g->V || p->V != g->V || p->B != (int32_t)s->batch_type.size())
        return fail(EDB_ERR_INVALID, "edb_prepare: graph, schedule and plan do not match");
    const int32_t T = g->T, B = p->B;
    std::vector<Dims> dims(T);
    int H = -1, E = -1, dtype = -1;
    for (int32_t t = 0; t < T; ++t) {
        edb_status st = cell_dims(&cells[t], dims[t]);
        if (st != EDB_OK) return fail(st, "edb_prepare: type " + std::to_string(t) + ": " + edb_last_error());
        if (H < 0) H = cells[t].hidden;
        if (cells[t].hidden != H) return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: all types must share hidden");
        if (dtype < 0) dtype = cells[t].dtype;
        if (cells[t].dtype != dtype) return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: all types must share dtype");
        if (kind_info(cells[t].kind).x) {   // types reading the caller's x
            if (E < 0) E = dims[t].E;
            if (dims[t].E != E) return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: all input types must share in_dim");
        }
        const KindInfo ki = kind_info(cells[t].kind);
        const edb_operand_shape& sh = p->shapes[t];
        if (sh.n_fixed != ki.nfix || (sh.ragged != 0) != ki.rag || (sh.has_x != 0) != ki.x)
            return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: operand shape of type " + std::to_string(t) +
                                                 " does not match its cell kind");
    }
    if (E < 0) E = 0;

    edb_exec* e = new (std::nothrow) edb_exec;
    if (!e) return fail(EDB_ERR_OOM, "edb_prepare: out of host memory");
    try {
        e->flags = flags;
        e->T = T;
        e->B = B;
        e->dtype = dtype;
        e->n_slots = p->n_slots;
        e->E = E;
        e->H = H;
        e->dims = dims;
        e->cells.assign(cells, cells + T);
        int n_x = 0;
        for (int32_t v = 0; v < g->V; ++v) {
            n_x += p->x_slot[v] >= 0;
            if (p->x_slot[v] >= 0) e->x_direct_rows = std::max(e->x_direct_rows, g->x_row[v] + 1);
        }
        e->n_x = n_x;
        // Staging x is skipped where it would only move rows around.  When every
        // node's staged row is its own row of the caller's x, the batches read x
        // in place through the same contiguous segments.  When a single batch
        // reads x (a forest's leaf batch), it reads the caller's rows through its
        // row list, as under EDB_X_DIRECT.
        if (!(flags & EDB_X_DIRECT) && n_x > 0) {
            bool same = true;
            for (int32_t v = 0; v < g->V && same; ++v)
                if (p->x_slot[v] >= 0 && p->x_slot[v] != g->x_row[v]) same = false;
            int x_batches = 0;
            for (int32_t b = 0; b < B; ++b) x_batches += kind_info(cells[s->batch_type[b]].kind).x ? 1 : 0;
            if (same) e->x_in_place = true;
            else if (x_batches == 1) e->flags = flags = flags | EDB_X_DIRECT;
        }
        // the large tile addresses x and the arena with 32-bit byte offsets
        const int64_t esz_b = dtype == EDB_F32 ? 4 : 2;   // x element size
        const int64_t off_limit = (int64_t)1 << 31;
        const bool large_fits = (int64_t)p->n_slots * H * 4 + (1 << 20) < off_limit &&   // arena_c (and arena_h)
                                (int64_t)std::max(n_x, e->x_direct_rows) * std::max(E, 1) * esz_b + (1 << 20) < off_limit;

        // device int buffer: plan idx pool | ragged pool | x source rows | zero rows
        std::vector<int32_t>& hb = e->hbuf;
        hb.insert(hb.end(), p->idx_pool.begin(), p->idx_pool.end());
        const int64_t off_rag = (int64_t)hb.size();
        hb.insert(hb.end(), p->ragged_pool.begin(), p->ragged_pool.end());
        e->off_xsrc = (int64_t)hb.size();
        hb.resize(hb.size() + n_x, 0);
        for (int32_t v = 0; v < g->V; ++v)
            if (p->x_slot[v] >= 0) hb[e->off_xsrc + p->x_slot[v]] = g->x_row[v];
        e->off_zero = (int64_t)hb.size();
        hb.push_back(0);
        hb.insert(hb.end(), p->pads.begin(), p->pads.end());
        e->n_zero = 1 + (int32_t)p->pads.size();
        if (hb.empty()) hb.push_back(0);

        int max_lds = 160 * 1024, n_cu = 256;
        DeviceCtx* ctx = nullptr;
        if (!(flags & EDB_DRYRUN)) {
            int dev = 0;
            hipError_t he = hipGetDevice(&dev);
            if (he == hipSuccess) he = device_ctx(dev, &ctx);
            if (he != hipSuccess) {
                delete e;
                return fail(EDB_ERR_HIP, std::string("edb_prepare: ") + hipGetErrorString(he));
            }
            e->device = dev;
            max_lds = ctx->max_lds;
            n_cu = ctx->n_cu;
        }
        const int force_var = std::getenv("EDB_VARIANT") ? std::atoi(std::getenv("EDB_VARIANT")) : -1;
        // occupancy per (kernel, dynamic LDS): the device context's cache is
        // shared by every thread behind one lock, so each prepare keeps the
        // values it has looked up (a few dozen) in a list of its own
        std::vector<std::tuple<const void*, int, int>> occ_seen;
        const OccFn occ = [&](const Entry& en, int block, int dyn_lds, int lds) -> int {
            const int est = std::max(1, std::min({max_lds / std::max(lds, 1), 32 / std::max(block / 64, 1), 16}));
            if (!ctx || !en.fn) return est;
            for (const auto& o : occ_seen)
                if (std::get<0>(o) == en.fn && std::get<1>(o) == dyn_lds) return std::get<2>(o);
            int nb = 0;
            {
                std::lock_guard<std::mutex> lk(g_ctx_mu);
                const auto key = std::make_pair(en.fn, dyn_lds);
                auto it = ctx->occupancy.find(key);
                if (it != ctx->occupancy.end()) {
                    nb = it->second;
                } else {
                    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, en.fn, block, (size_t)dyn_lds) != hipSuccess ||
                        nb < 1) {
                        (void)hipGetLastError();
                        nb = est;
                    }
                    ctx->occupancy[key] = nb;
                }
            }
            occ_seen.emplace_back(en.fn, dyn_lds, nb);
            return nb;
        };

        // launch 0: x staging + zero rows
        {
            Launch L{};
            L.info.batch = -1;
            L.info.kind = -1;
            L.info.m = n_x;
            L.info.grid = (((flags & EDB_X_DIRECT) || e->x_in_place ? 0 : n_x) + e->n_zero + 3) / 4;   // 4 rows per work-group
            L.info.block = 256;
            L.info.variant = -1;
            L.info.n_batches = 0;
            e->launches.push_back(L);
        }
        const bool force_gather = (flags & EDB_FORCE_GATHER) != 0;
        std::vector<std::vector<Launch>> blaunch;   // the launches of each batch, in order
        blaunch.reserve(B);
        for (int32_t b = 0; b < B; ++b) {
            const int32_t t = s->batch_type[b];
            const Dims& d = dims[t];
            const int32_t m = s->batch_ptr[b + 1] - s->batch_ptr[b];
            const int32_t* ord = p->order.data() + s->batch_ptr[b];
            Launch L{};
            L.type = t;
            L.info.batch = b;
            L.info.kind = cells[t].kind;
            L.info.m = m;
            L.info.k = d.K;
            L.info.n = d.G * d.Hu;
            L.info.block = 256;
            L.off_x = L.off_f0 = L.off_f1 = L.off_rag = L.off_rptr = L.off_res = -1;
            BatchArgs& a = L.args;
            a.kind = cells[t].kind;
            a.m = m;
            a.H = d.H;
            a.Hk = d.Hk;
            a.Hu = d.Hu;
            a.E = d.E;
            a.Ep = d.Ep;
            a.K = d.K;
            // segments of this batch: result, positional lists, ragged list
            const edb_seg* sg = p->segs.data() + p->seg_ptr[b];
            auto conv = [&](const edb_seg& q, Seg& out_seg, int64_t& off) {
                off = -1;
                out_seg = Seg{S_NONE, 0, nullptr};
                if (q.kind == EDB_SEG_NONE) return;
                if (q.kind == EDB_SEG_CONTIG && !force_gather) {
                    out_seg.kind = S_CONTIG;
                    out_seg.base = q.base;
                } else {
                    out_seg.kind = S_INDEXED;
                    off = q.idx_off;
                }
            };
            conv(sg[0], a.res, L.off_res);
            L.info.seg_kind[0] = sg[0].kind;
            const KindInfo ki = kind_info(cells[t].kind);
            if (ki.nfix >= 1) { conv(sg[1], a.fix[0], L.off_f0); L.info.seg_kind[1] = sg[1].kind; }
            if (ki.nfix >= 2) { conv(sg[2], a.fix[1], L.off_f1); L.info.seg_kind[2] = sg[2].kind; }
            if (ki.rag) {
                conv(sg[1 + ki.nfix], a.rag, L.off_rag);
                L.info.seg_kind[3] = sg[1 + ki.nfix].kind;
                L.off_rptr = off_rag + p->ragged_off[b];
                // rag_ptr entries are offsets into this batch's ragged list
            }
            if (ki.x) {
                const int xb = p->x_slot[ord[0]];
                if (flags & EDB_X_DIRECT) {
                    a.x = Seg{S_INDEXED, 0, nullptr};
                    L.off_x = e->off_xsrc + xb;
                } else {
                    a.x = Seg{S_CONTIG, xb, nullptr};
                }
            }
            // tile variant: smallest estimated time under a simple model (matrix
            // core cycles of the busiest SIMD plus per-k-group latency), ties
            // to the larger tile; variants whose LDS need exceeds the device
            // limit are skipped
            const int kind_id = cells[t].kind;
            L.kk = kind_id;
            int var = -1;
            double best = 1e300;
            // the large tile reads whole 64-wide k chunks of one operand segment
            const int big_chunk = dtype == EDB_F32 ? 32 : 64;   // k values per 128-byte chunk
            const bool large_ok = large_fits && d.Ep % big_chunk == 0 && d.Hk % big_chunk == 0 && !(flags & EDB_NO_LARGE);
            const bool cs_large = kind_id == EDB_CELL_CS_INTERNAL && dtype == EDB_BF16;
            const int64_t nrag = d.rag ? p->ragged_pool[p->ragged_off[b] + m] : 0;   // children of the batch
            // large tile: the cell's own kernel, or for child-sum cells the
            // child sums, the forget GEMM over the children and the parents
            int lvar = -1, fvar = -1;
            double lest = 1e300;
            if (large_ok && cs_large) {
                if (nrag > 0 && nrag * (int64_t)d.H * 4 + (1 << 20) < ((int64_t)1 << 31)) {
                    double ef = 0, ep = 0;
                    fvar = best_large(K_CS_FORGET, dtype, 1, (int)nrag, d.K, d.Hu, n_cu, max_lds, occ, ef);
                    lvar = best_large(K_CS_PARENT, dtype, 3, m, d.K, d.Hu, n_cu, max_lds, occ, ep);
                    if (fvar < 0 || lvar < 0) lvar = fvar = -1;
                    else lest = ef + ep + child_reduce_cost(m);
                }
            } else if (large_ok) {
                lvar = best_large(kind_id, dtype, d.G, m, d.K, d.Hu, n_cu, max_lds, occ, lest);
            }
            const bool large_only = (flags & EDB_TILE_LARGE) && lvar >= 0;
            for (int vi = 0; vi < NUM_VARIANTS && !large_only; ++vi) {
                if (!is_small(vi) && !(is_stream(vi) && large_fits)) continue;
                const Entry& en = table().e[kind_id][dtype][vi];
                if (!en.fn) continue;
                const int lds = en.lds(d.K, d.Hk);
                if (lds > max_lds) continue;
                if (d.rag && VAR_WU[vi] * VAR_WK[vi] > 8) continue;   // register budget of 1024 threads
                if ((flags & EDB_NO_SPLIT_K) && VAR_WK[vi] != 1) continue;
                const int block = 64 * VAR_WU[vi] * VAR_WK[vi];
                const double est = variant_cost(vi, m, d, dtype, nrag, occ(en, block, lds, lds), n_cu);
                if (est < best * 0.97) { best = est; var = vi; }
            }
            // the large tile where its estimate beats the small and streamed tiles'
            if (lvar >= 0 && (large_only || var < 0 || lest < best)) var = lvar;
            // a forced streamed variant falls back to its staged counterpart
            // for kinds it does not serve (and buffers beyond 32-bit offsets)
            int fv = force_var;
            if (is_stream(fv) && !(large_fits && table().e[kind_id][dtype][fv].fn))
                fv = STAGED_OF[fv - FIRST_STREAM];
            if ((is_small(fv) || is_stream(fv)) && table().e[kind_id][dtype][fv].fn &&
                table().e[kind_id][dtype][fv].lds(d.K, d.Hk) <= max_lds)
                var = fv;
            if (is_large(force_var) && lvar >= 0) {
                const int fk = cs_large ? K_CS_PARENT : kind_id;
                if (table().e[fk][dtype][force_var].fn) var = lvar = force_var;
                if (cs_large && table().e[K_CS_FORGET][dtype][force_var].fn) fvar = force_var;
            }
            // the weight-stationary tile for the largest x-only batches (bf16):
            // the weights of its 32 units and its row table fit the LDS, the
            // reduction is a whole number of the ring's groups of k-groups, at
            // least two (the ring then reaches at most one tile ahead), and
            // offsets stay 32-bit
            {
                const Entry& wen = table().e[kind_id][dtype][WS_VARIANT];
                const bool ws_ok = wen.fn && !cs_large && large_fits && !(flags & EDB_NO_LARGE) &&
                                   d.K % (32 * WS_D) == 0 && d.K / 32 >= 2 * WS_D &&
                                   d.Hu % WS_TU == 0 && wen.lds(d.K, d.Hk) <= max_lds;
                if (ws_ok && ((m >= kWsMinRows && force_var < 0) || force_var == WS_VARIANT)) var = WS_VARIANT;
            }
            if (var < 0) {
                delete e;
                return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: no tile variant fits the LDS of batch " +
                                                     std::to_string(b));
            }
            std::vector<Launch> parts;
            if (kind_id == EDB_CELL_MV_VEC) {
                // 1: the matrix-vector products [B a, A b] of every row into
                // the mvu scratch, then 0: the GEMM with those rows as x
                const int64_t ro = p->ragged_off[b];
                for (int32_t r = 0; r < m; ++r)
                    if (p->ragged_pool[ro + r + 1] - p->ragged_pool[ro + r] != 2 * d.H) {
                        delete e;
                        return fail(EDB_ERR_INVALID, "edb_prepare: an MV_VEC node of batch " + std::to_string(b) +
                                                         " does not list exactly 2 * hidden matrix columns");
                    }
                Launch C = L;
                C.kk = -2;
                C.lds = 0;
                C.info.part = 1;
                C.info.variant = -1;
                C.info.n_batches = 0;
                C.info.k = 0;
                C.info.n = 2 * d.H;
                C.info.block = 256;
                C.info.grid = (2 * m + 3) / 4;
                parts.push_back(C);
                L.args.x = Seg{S_CONTIG, 0, nullptr};
                L.off_x = -1;
                e->mvu_rows = std::max<int64_t>(e->mvu_rows, m);
            }
            if (is_large(var) && cs_large) {
                // 2: forget GEMM over the batch's children (rows: the child list): sigma(f_k) c_k
                Launch F = L;
                F.kk = K_CS_FORGET;
                F.info.part = 2;
                F.info.variant = fvar;
                F.info.n_batches = 0;
                F.info.m = (int)nrag;
                F.info.k = d.K;
                F.info.n = d.Hu;
                F.args.kind = K_CS_FORGET;
                F.args.m = (int)nrag;
                F.args.x = L.args.rag;
                F.off_x = L.off_rag;
                F.args.E = d.H;
                F.args.Ep = d.Hk;
                F.args.res = Seg{S_NONE, 0, nullptr};
                F.off_res = -1;
                F.lds = table().e[K_CS_FORGET][dtype][fvar].lds(d.K, d.Hk);
                F.info.block = 256;
                F.info.grid = ((int)((nrag + large_tm(1, large_class(fvar)) - 1) / large_tm(1, large_class(fvar))) *
                                   (d.Hu / large_tu(large_class(fvar))) + 7) / 8 * 8;
                parts.push_back(F);
                // 1: per parent, the child sum of h (h~) and the sum of the children's products
                Launch C = L;
                C.kk = -1;
                C.lds = 0;
                C.info.part = 1;
                C.info.variant = -1;
                C.info.n_batches = 0;
                C.info.k = 0;
                C.info.n = d.H;
                C.info.block = 256;
                C.info.grid = (int)(((int64_t)m * (d.H / 8) + 255) / 256);
                parts.push_back(C);
                // 0: the parents on their child sums (their children's products summed)
                L.kk = K_CS_PARENT;
                L.args.kind = K_CS_PARENT;
                L.args.x = Seg{S_CONTIG, 0, nullptr};
                L.off_x = -1;
                L.args.E = d.H;
                L.args.Ep = d.Hk;
                e->hsum_rows = std::max<int64_t>(e->hsum_rows, m);
                e->fc_rows = std::max<int64_t>(e->fc_rows, nrag);
            }
            L.lds = table().e[L.kk][dtype][var].lds(d.K, d.Hk);
            if (L.lds > max_lds) {
                delete e;
                return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: LDS need of batch " + std::to_string(b) +
                                                     " exceeds the device limit");
            }
            L.info.variant = var;
            L.info.n_batches = 1;
            L.info.part = 0;
            if (is_ws(var)) {
                // unit tiles x row groups, the row groups a multiple of 8 (one XCD
                // holds whole row groups), about one work-group per CU, and at
                // most WS_MAXT row tiles per work-group (its row table)
                const int nut = d.Hu / WS_TU;
                const int nrt = (m + WS_TM - 1) / WS_TM;
                const int need = (nrt + WS_MAXT - 1) / WS_MAXT;
                const int ngr = std::max({8, std::min((n_cu / nut) / 8 * 8, (nrt + 7) / 8 * 8), (need + 7) / 8 * 8});
                L.info.grid = nut * ngr;
                L.info.block = WS_NT;
            } else if (is_large(var)) {
                const int TM = large_tm(d.G, large_class(var));
                const int tiles = (m + TM - 1) / TM * (d.Hu / large_tu(large_class(var)));
                L.info.grid = (tiles + 7) / 8 * 8;   // XCD-aware order: 8 equal tile ranges
                L.info.block = 256;
            } else if (is_stream(var)) {
                const int TM = 16 * VAR_RT[var];
                const int tiles = (m + TM - 1) / TM * (d.Hu / 16);
                L.info.grid = (tiles + 7) / 8 * 8;   // XCD-aware order: 8 equal tile ranges
                L.info.block = 64 * VAR_WK[var];
            } else {
                const int TM = 16 * VAR_RT[var], TU = 16 * VAR_WU[var];
                L.info.grid = (m + TM - 1) / TM * (d.Hu / TU);
                L.info.block = 64 * VAR_WU[var] * VAR_WK[var];
            }
            parts.push_back(L);
            blaunch.push_back(std::move(parts));
        }

        // ---- dataflow runs: maximal runs (>= 2) of consecutive batches with at
        // most flow_max_m rows each are executed by one persistent launch ----
        int flow_max_m = 1024;
        if (const char* ev = std::getenv("EDB_FLOW_MAX_M")) flow_max_m = std::atoi(ev);
        int spin_us = 100000;   // bound of one tile's dependency wait (microseconds)
        if (const char* ev = std::getenv("EDB_SPIN_US")) spin_us = std::max(1, std::atoi(ev));
        // Dataflow launches are switched off: their first GPU runs did not
        // finish (the launch did not drain within minutes although every wait
        // is bounded in time); until the cause is shown, every batch runs as
        // its own launch.  The code below stays for that analysis.
        constexpr bool kFlowEnabled = false;
        const bool flow_on = (kFlowEnabled || (flags & EDB_FLOW_DRYRUN)) && !(flags & EDB_NO_FLOW) &&
                             T <= FLOW_MAX_TYPES && flow_max_m > 0;
        std::vector<int> run_of(B, -1);
        {
            int b = 0, nrun = 0;
            while (b < B) {
                const int m0 = s->batch_ptr[b + 1] - s->batch_ptr[b];
                // the dataflow kernel serves the kinds up to TreeGRU
                auto flow_ok = [&](int q) { return blaunch[q].size() == 1 && blaunch[q][0].kk <= K_GRU_INT; };
                if (!flow_on || m0 > flow_max_m || !flow_ok(b)) { ++b; continue; }
                int b1 = b;
                while (b1 < B && s->batch_ptr[b1 + 1] - s->batch_ptr[b1] <= flow_max_m && flow_ok(b1)) ++b1;
                if (b1 - b >= 2) {
                    for (int q = b; q < b1; ++q) run_of[q] = nrun;
                    ++nrun;
                }
                b = b1;
            }
        }
        // row of every node inside its batch (for dependency lists)
        std::vector<int32_t> node_batch(g->V, -1), node_row(g->V, -1);
        for (int32_t b = 0; b < B; ++b)
            for (int32_t i = s->batch_ptr[b]; i < s->batch_ptr[b + 1]; ++i) {
                node_batch[p->order[i]] = b;
                node_row[p->order[i]] = i - s->batch_ptr[b];
            }
        auto align_hb = [&](int a) { while (hb.size() % a) hb.push_back(0); };
        std::vector<int64_t> counter_fix;   // launches whose counter offsets need the final base
        int64_t n_counters = 0;
        for (int32_t b = 0; b < B;) {
            if (run_of[b] < 0) {
                for (const Launch& Lp : blaunch[b]) e->launches.push_back(Lp);
                ++b;
                continue;
            }
            int b1 = b;
            while (b1 < B && run_of[b1] == run_of[b]) ++b1;
            Launch F{};
            F.flow = true;
            F.info.batch = b;
            F.info.kind = -1;
            F.info.variant = FLOW_VARIANT;
            F.info.n_batches = b1 - b;
            F.info.block = 64 * FLOW_WU * FLOW_WK;
            F.info.k = 0;
            F.info.n = 0;
            // batch descriptors
            align_hb(4);
            F.f_desc = (int64_t)hb.size();
            std::vector<int> kinds_k;
            for (int q = b; q < b1; ++q) {
                const Launch& L = blaunch[q].back();
                const Dims& d = dims[L.type];
                BatchDesc bd{};
                bd.kind = L.info.kind;
                bd.type = L.type;
                bd.m = L.args.m;
                bd.H = d.H; bd.Hk = d.Hk; bd.Hu = d.Hu; bd.E = d.E; bd.Ep = d.Ep; bd.K = d.K;
                bd.x_staged = (flags & EDB_X_DIRECT) || e->x_in_place ? 0 : 1;
                const Seg* sgs[5] = {&L.args.x, &L.args.fix[0], &L.args.fix[1], &L.args.rag, &L.args.res};
                const int64_t offs[5] = {L.off_x, L.off_f0, L.off_f1, L.off_rag, L.off_res};
                for (int i = 0; i < 5; ++i) {
                    bd.seg_kind[i] = sgs[i]->kind;
                    bd.seg_base[i] = sgs[i]->base;
                    bd.seg_off[i] = (int)offs[i];
                }
                bd.rptr_off = (int)L.off_rptr;
                bd.off_b = (int)d.off_b;
                bd.off_Wr = (int)d.off_Wr;
                bd.off_br = (int)d.off_br;
                const int32_t* bw = reinterpret_cast<const int32_t*>(&bd);
                hb.insert(hb.end(), bw, bw + sizeof(BatchDesc) / 4);
                F.info.m += bd.m;
                kinds_k.push_back(bd.kind);
                kinds_k.push_back(bd.K);
            }
            // row tiles and their producer row tiles inside the run
            std::vector<int> rt_base(b1 - b + 1, 0);
            const int nut = dims[blaunch[b].back().type].Hu / (16 * FLOW_WU);
            for (int q = b; q < b1; ++q)
                rt_base[q - b + 1] = rt_base[q - b] + (blaunch[q].back().args.m + 16 * FLOW_RT - 1) / (16 * FLOW_RT);
            const int nrt = rt_base[b1 - b];
            std::vector<int32_t> rtdeps(2 * nrt), deps, tmp;
            for (int q = b; q < b1; ++q) {
                const int32_t* ord = p->order.data() + s->batch_ptr[q];
                const int m = blaunch[q].back().args.m;
                for (int rt = 0; rt * 16 * FLOW_RT < m; ++rt) {
                    tmp.clear();
                    for (int r = rt * 16 * FLOW_RT; r < std::min(m, (rt + 1) * 16 * FLOW_RT); ++r) {
                        const int32_t v = ord[r];
                        for (int64_t k = g->child_ptr[v]; k < g->child_ptr[v + 1]; ++k) {
                            const int32_t c = g->child_idx[k];
                            if (c < 0) continue;
                            const int cb = node_batch[c];
                            if (cb < b || cb >= b1) continue;   // produced by an earlier launch
                            tmp.push_back(rt_base[cb - b] + node_row[c] / (16 * FLOW_RT));
                        }
                    }
                    std::sort(tmp.begin(), tmp.end());
                    tmp.erase(std::unique(tmp.begin(), tmp.end()), tmp.end());
                    const int id = rt_base[q - b] + rt;
                    rtdeps[2 * id] = (int32_t)deps.size();
                    rtdeps[2 * id + 1] = (int32_t)tmp.size();
                    deps.insert(deps.end(), tmp.begin(), tmp.end());
                }
            }
            align_hb(4);
            F.f_tiles = (int64_t)hb.size();
            for (int q = b; q < b1; ++q) {
                const int m = blaunch[q].back().args.m;
                for (int rt = 0; rt * 16 * FLOW_RT < m; ++rt)
                    for (int ut = 0; ut < nut; ++ut) {
                        hb.push_back(q - b);
                        hb.push_back(rt);
                        hb.push_back(ut);
                        hb.push_back(rt_base[q - b] + rt);
                        ++F.f_ntiles;
                    }
            }
            align_hb(2);
            F.f_rtdeps = (int64_t)hb.size();
            hb.insert(hb.end(), rtdeps.begin(), rtdeps.end());
            F.f_deps = (int64_t)hb.size();
            hb.insert(hb.end(), deps.begin(), deps.end());
            if (deps.empty()) hb.push_back(0);
            // counters (offsets relative to the counter region, fixed below)
            F.f_ticket = n_counters;
            F.f_error = n_counters + 1;
            F.f_done = n_counters + 2;
            n_counters += 2 + nrt;
            F.f_need = nut;
            F.info.grid = F.f_ntiles;   // capped by occupancy below
            F.lds = dtype == EDB_F32 ? flow_lds<float>(kinds_k) : flow_lds<__bf16>(kinds_k);
            F.args.m = spin_us;          // carried to execute
            counter_fix.push_back((int64_t)e->launches.size());
            e->launches.push_back(F);
            b = b1;
        }
        // counter region: zeroed by the staging kernel before every forward
        align_hb(4);
        e->off_counters = (int64_t)hb.size();
        e->n_counters = n_counters;
        hb.resize(hb.size() + n_counters, 0);
        for (int64_t li : counter_fix) {
            Launch& F = e->launches[li];
            F.f_ticket += e->off_counters;
            F.f_error += e->off_counters;
            F.f_done += e->off_counters;
        }
        // When the staging launch would only clear the zero and pad rows, the
        // first batch's launch clears them and the staging launch is dropped
        // (grid 0).  Only for a first batch without child lists (it then reads
        // no arena row) whose x segment has no padding columns (the staged
        // tile reads the zero row for those), run as a single launch.
        if (e->launches.size() > 1 && n_counters == 0) {
            Launch& L1 = e->launches[1];
            const bool staged_x = !((flags & EDB_X_DIRECT) || e->x_in_place) && n_x > 0;
            const KindInfo k1 = L1.flow ? KindInfo{} : kind_info(L1.info.kind);
            const bool single = !L1.flow && L1.info.batch == 0 && L1.info.part == 0 && L1.kk == L1.info.kind &&
                                (e->launches.size() == 2 || e->launches[2].info.batch != 0);
            if (!staged_x && single && k1.G > 0 && k1.nfix == 0 && !k1.rag && dims[L1.type].Ep == dims[L1.type].E) {
                e->launches[0].info.grid = 0;
                L1.off_zrows = e->off_zero;
                L1.args.n_zero = e->n_zero;
            }
        }
        // dataflow grids: at most the resident work-groups (more would only exit)
        for (Launch& F : e->launches) {
            if (!F.flow) continue;
            if (F.lds > max_lds) {
                delete e;
                return fail(EDB_ERR_UNSUPPORTED, "edb_prepare: dataflow LDS need exceeds the device limit");
            }
            int resident = 512;
            if (!(flags & EDB_DRYRUN)) {
                const void* fn = dtype == EDB_F32 ? reinterpret_cast<const void*>(&flow_kernel<float>)
                                                  : reinterpret_cast<const void*>(&flow_kernel<__bf16>);
                hipError_t he = hipSuccess;
                if (F.lds > 64 * 1024) {
                    std::lock_guard<std::mutex> lk(g_ctx_mu);
                    int& granted = ctx->lds_granted[-1 - dtype];
                    if (F.lds > granted) {
                        he = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, F.lds);
                        if (he == hipSuccess) granted = F.lds;
                    }
                }
                int nb = 0;
                if (he == hipSuccess) he = hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, 256, F.lds);
                if (he != hipSuccess) {
                    delete e;
                    return fail(EDB_ERR_HIP, std::string("edb_prepare: ") + hipGetErrorString(he));
                }
                resident = std::max(1, nb) * ctx->n_cu;
            }
            F.info.grid = std::max(1, std::min(F.f_ntiles, resident));
        }

        layout_device(e);
        if (!(flags & EDB_DRYRUN)) {
            // descriptors and the staged-x buffer: one stream-ordered allocation
            // on the upload stream, filled asynchronously; executions wait on
            // the `ready` event instead of the host waiting for the copy
            hipError_t he = noalloc ? hipSuccess : ctx_streams(ctx);
            if (!noalloc && he == hipSuccess) {
                e->upload = ctx->upload;
                e->release = ctx->release;
                he = hipMallocAsync(&e->dmem, e->d_total, ctx->upload);
                if (he != hipSuccess) {
                    (void)hipGetLastError();
                    e->dmem = nullptr;
                    e->dmem_async = false;
                    he = hipMalloc(&e->dmem, e->d_total);
                }
                if (he == hipSuccess) {
                    bind_device(e, e->dmem);
                    he = hipMemcpyAsync(e->dbuf, hb.data(), hb.size() * sizeof(int32_t), hipMemcpyHostToDevice,
                                        ctx->upload);
                }
                if (he == hipSuccess) he = hipEventCreateWithFlags(&e->ready, hipEventDisableTiming);
                if (he == hipSuccess) he = hipEventCreateWithFlags(&e->done, hipEventDisableTiming);
                if (he == hipSuccess) he = hipEventRecord(e->ready, ctx->upload);
            }
            if (!noalloc && (flags & EDB_PROFILE)) {
                e->ctx = ctx;
                e->events.assign(2 * e->launches.size(), nullptr);
                {
                    std::lock_guard<std::mutex> lk(g_ctx_mu);
                    for (size_t i = 0; i < e->events.size() && !ctx->event_pool.empty(); ++i) {
                        e->events[i] = ctx->event_pool.back();
                        ctx->event_pool.pop_back();
                    }
                }
                for (size_t i = 0; he == hipSuccess && i < e->events.size(); ++i)
                    if (!e->events[i]) he = hipEventCreate(&e->events[i]);
            }
            for (size_t i = 1; he == hipSuccess && i < e->launches.size(); ++i) {
                const Launch& L = e->launches[i];
                if (L.lds <= 64 * 1024 || L.flow || L.kk < 0) continue;
                const int key = (L.kk * 2 + dtype) * NUM_VARIANTS + L.info.variant;
                std::lock_guard<std::mutex> lk(g_ctx_mu);
                int& granted = ctx->lds_granted[key];
                if (L.lds > granted) {
                    he = table().e[L.kk][dtype][L.info.variant].attr(L.lds);
                    if (he == hipSuccess) granted = L.lds;
                }
            }
            if (he != hipSuccess) {
                const bool oom = he == hipErrorOutOfMemory;
                delete e;
                return fail(oom ? EDB_ERR_OOM : EDB_ERR_HIP, std::string("edb_prepare: ") + hipGetErrorString(he));
            }
        }
    } catch (const std::bad_alloc&) {
        delete e;
        return fail(EDB_ERR_OOM, "edb_prepare: out of host memory");
    }
    edb::clear_error();
    *out = e;
    return EDB_OK;
}

// Launch L's arguments with the pointers of one execution filled in (w may be
// NULL when no weights are read).
BatchArgs resolve_args(const edb_exec* e, const Launch& L, const void* const* w, const void* x, void* arena_h,
                       void* arena_c) {
    const int* db = e->dbuf;
    BatchArgs a = L.args;
    const Dims& d = e->dims[L.type];
    if (w) {
        const uint8_t* wb = reinterpret_cast<const uint8_t*>(w[L.type]);
        a.W = wb + d.off_W;
        a.bias = reinterpret_cast<const float*>(wb + d.off_b);
        a.Wr = d.rag ? wb + d.off_Wr : nullptr;
        a.br = d.rag ? reinterpret_cast<const float*>(wb + d.off_br) : nullptr;
    }
    a.arena_h = arena_h;
    a.arena_c = reinterpret_cast<float*>(arena_c);
    const bool x_caller = (e->flags & EDB_X_DIRECT) || e->x_in_place;
    a.xmat = x_caller ? x : e->xstaged;
    a.n_slots = e->n_slots;
    a.n_xrows = x_caller ? e->x_direct_rows : e->n_x;
    a.fc = e->fc;
    if (L.off_x >= 0) a.x.idx = db + L.off_x;
    if (L.off_f0 >= 0) a.fix[0].idx = db + L.off_f0;
    if (L.off_f1 >= 0) a.fix[1].idx = db + L.off_f1;
    if (L.off_rag >= 0) a.rag.idx = db + L.off_rag;
    if (L.off_rptr >= 0) a.rag_ptr = db + L.off_rptr;
    if (L.off_res >= 0) a.res.idx = db + L.off_res;
    if (L.off_zrows >= 0) a.zrows = db + L.off_zrows;
    return a;
}

// One kernel call of an execution: the kernel, its launch shape and its
// arguments by value.  The same list is issued eagerly or written into the
// nodes of a HIP graph, so both ways run the same calls.
struct Call {
    const void* fn = nullptr;
    unsigned grid = 0, block = 256;
    size_t lds = 0;               // dynamic LDS bytes
    int launch = 0;               // its launch record (EDB_PROFILE events)
    int form = 0;                 // 0 (BatchArgs), 1 (BatchArgs, bf16*, float*), 2 (BatchArgs, T*), 3 staging, 4 dataflow
    BatchArgs a{};
    void* p0 = nullptr;
    void* p1 = nullptr;
    FlowArgs f{};
    struct Stage {                // stage_kernel's parameters, in order
        const void* x;
        void* xs;
        const int* src;
        int n_x, E;
        const int* zrow;
        int n_zero;
        void* arena_h;
        float* arena_c;
        int H;
        int* ints;
        int nint;
    } s{};
    void* argv[12];
    // pointers to the arguments (into this object: call after it has its final address)
    void** args() {
        switch (form) {
            case 0: argv[0] = &a; break;
            case 1: argv[0] = &a; argv[1] = &p0; argv[2] = &p1; break;
            case 2: argv[0] = &a; argv[1] = &p0; break;
            case 3:
                argv[0] = &s.x; argv[1] = &s.xs; argv[2] = &s.src; argv[3] = &s.n_x; argv[4] = &s.E;
                argv[5] = &s.zrow; argv[6] = &s.n_zero; argv[7] = &s.arena_h; argv[8] = &s.arena_c;
                argv[9] = &s.H; argv[10] = &s.ints; argv[11] = &s.nint;
                break;
            default: argv[0] = &f; break;
        }
        return argv;
    }
};

// The calls of one execution, in launch order (records with grid 0 are not issued).
void build_calls(const edb_exec* e, const void* const* w, const void* x, void* arena_h, void* arena_c,
                 std::vector<Call>& out) {
    out.clear();
    out.reserve(e->launches.size());
    const int* db = e->dbuf;
    const bool f32 = e->dtype == EDB_F32;
    // launch 0: stage x rows, clear the zero / pad rows and the dataflow counters
    {
        const Launch& L = e->launches[0];
        const bool direct = (e->flags & EDB_X_DIRECT) != 0 || e->x_in_place;
        if (L.info.grid > 0) {
            Call c;
            c.fn = f32 ? reinterpret_cast<const void*>(&stage_kernel<float>)
                       : reinterpret_cast<const void*>(&stage_kernel<__bf16>);
            c.grid = L.info.grid;
            c.form = 3;
            c.s = Call::Stage{x, e->xstaged, db + e->off_xsrc, direct ? 0 : e->n_x, e->E, db + e->off_zero,
                              e->n_zero, arena_h, reinterpret_cast<float*>(arena_c), e->H,
                              e->dbuf + e->off_counters, (int)e->n_counters};
            out.push_back(c);
        }
    }
    for (size_t i = 1; i < e->launches.size(); ++i) {
        const Launch& L = e->launches[i];
        if (L.info.grid <= 0) continue;
        Call c;
        c.launch = (int)i;
        c.grid = L.info.grid;
        if (L.flow) {
            FlowArgs& f = c.f;
            f.ibuf = db;
            f.desc = reinterpret_cast<const BatchDesc*>(db + L.f_desc);
            f.tiles = reinterpret_cast<const int4*>(db + L.f_tiles);
            f.rt_deps = reinterpret_cast<const int2*>(db + L.f_rtdeps);
            f.deps = db + L.f_deps;
            f.ticket = e->dbuf + L.f_ticket;
            f.error = e->dbuf + L.f_error;
            f.done = e->dbuf + L.f_done;
            f.n_tiles = L.f_ntiles;
            f.need = L.f_need;
            f.spin_us = L.args.m;
            f.n_slots = e->n_slots;
            f.n_xrows = (e->flags & EDB_X_DIRECT) || e->x_in_place ? e->x_direct_rows : e->n_x;
            f.x = x;
            f.xstaged = e->xstaged;
            f.arena_h = arena_h;
            f.arena_c = reinterpret_cast<float*>(arena_c);
            for (int t = 0; t < e->T && t < FLOW_MAX_TYPES; ++t) f.w[t] = w[t];
            c.fn = f32 ? reinterpret_cast<const void*>(&flow_kernel<float>)
                       : reinterpret_cast<const void*>(&flow_kernel<__bf16>);
            c.lds = L.lds;
            c.form = 4;
            out.push_back(c);
            continue;
        }
        c.a = resolve_args(e, L, w, x, arena_h, arena_c);
        if (L.kk == -2) {   // MV-RNN vector batch: [B a, A b] into the mvu scratch (fp32 only)
            c.fn = reinterpret_cast<const void*>(&mv_matvec_kernel<float>);
            c.form = 2;
            c.p0 = e->mvu;
            out.push_back(c);
            continue;
        }
        if (L.kk < 0) {   // child-sum batch on the large tile: child sums and product sums
            c.fn = reinterpret_cast<const void*>(&child_reduce_kernel);
            c.form = 1;
            c.p0 = e->hsum;
            c.p1 = e->racc;
            out.push_back(c);
            continue;
        }
        BatchArgs& a = c.a;
        if (L.kk == K_CS_FORGET) {   // rows: the children's h; weights U_f, b_f
            a.W = a.Wr;
            a.bias = a.br;
            a.xmat = arena_h;
            a.n_xrows = e->n_slots;
        } else if (L.kk == K_MV_VEC) {   // rows: [B a, A b] from the matrix-vector launch
            a.xmat = e->mvu;
            a.n_xrows = a.m;
        } else if (L.kk == K_CS_PARENT) {   // rows: the child sums; epilogue: the product sums
            a.xmat = e->hsum;
            a.n_xrows = a.m;
            a.fc = e->racc;
        }
        c.fn = table().e[L.kk][e->dtype][L.info.variant].fn;
        c.block = L.info.block;
        c.lds = is_large(L.info.variant) ? 0 : L.lds;   // the large tile's LDS is static
        out.push_back(c);
    }
}

hipError_t launch_all(edb_exec* e, const void* const* w, const void* x, void* arena_h, void* arena_c,
                      hipStream_t st) {
    thread_local std::vector<Call> calls;
    build_calls(e, w, x, arena_h, arena_c, calls);
    const bool prof = !e->events.empty();
    hipError_t he = hipSuccess;
    for (Call& c : calls) {
        if (prof)
            he = hipExtLaunchKernel(c.fn, dim3(c.grid), dim3(c.block), c.args(), c.lds, st, e->events[2 * c.launch],
                                    e->events[2 * c.launch + 1], 0);
        else
            he = hipLaunchKernel(c.fn, dim3(c.grid), dim3(c.block), c.args(), c.lds, st);
        if (he != hipSuccess) return he;
    }
    return hipGetLastError();
}

// Instantiated graphs of kernel-call sequences, kept per device and stream
// and reused by every later execution there whose sequence has the same
// kernels and block sizes: a new input graph updates the nodes' arguments,
// grids and LDS in place and is not instantiated again.  Up to kTopoPerStream
// sequences per stream; the least recently used one is replaced.  Kept for
// the life of the process.
constexpr int kTopoPerStream = 4;
struct Topo {
    std::vector<std::pair<const void*, unsigned>> sig;   // kernel and block size of each node
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    std::vector<hipGraphNode_t> nodes;
    hipEvent_t done = nullptr;     // after its last launch
    uint64_t used = 0;
    uint64_t owner = 0;            // executor (id) and pointers the nodes hold now
    std::vector<const void*> owner_ptrs;
};
struct TopoSet {
    std::mutex mu;
    std::vector<Topo> t;
    uint64_t tick = 0;
};
std::mutex g_topo_mu;
std::map<std::pair<int, hipStream_t>, TopoSet*> g_topo;
std::atomic<int64_t> g_topo_instantiated{0}, g_topo_updated{0};

hipKernelNodeParams node_params(Call& c) {
    hipKernelNodeParams p{};
    p.func = const_cast<void*>(c.fn);
    p.gridDim = dim3(c.grid);
    p.blockDim = dim3(c.block);
    p.sharedMemBytes = (unsigned)c.lds;
    p.kernelParams = c.args();
    p.extra = nullptr;
    return p;
}

// Runs the execution's calls on st through the stream's graph of the same
// kernel sequence (instantiated on first use).
hipError_t graph_launch(edb_exec* e, const void* const* w, const void* x, void* arena_h, void* arena_c,
                        hipStream_t st) {
    int dev = 0;
    hipError_t he = hipGetDevice(&dev);
    if (he != hipSuccess) return he;
    TopoSet* ts = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_topo_mu);
        TopoSet*& slot = g_topo[{dev, st}];
        if (!slot) slot = new TopoSet;
        ts = slot;
    }
    std::vector<const void*> ptrs(w, w + e->T);
    ptrs.push_back(x);
    ptrs.push_back(arena_h);
    ptrs.push_back(arena_c);
    ptrs.push_back(e->dbuf);
    thread_local std::vector<Call> calls;
    build_calls(e, w, x, arena_h, arena_c, calls);
    std::vector<std::pair<const void*, unsigned>> sig;
    sig.reserve(calls.size());
    for (const Call& c : calls) sig.emplace_back(c.fn, c.block);
    std::lock_guard<std::mutex> lk(ts->mu);
    Topo* t = nullptr;
    for (Topo& q : ts->t)
        if (q.sig == sig) { t = &q; break; }
    if (t) {
        // the same executor with the same buffers: the nodes already hold its calls
        if (t->owner != e->id || t->owner_ptrs != ptrs) {
            for (size_t i = 0; he == hipSuccess && i < calls.size(); ++i) {
                const hipKernelNodeParams np = node_params(calls[i]);
                he = hipGraphExecKernelNodeSetParams(t->exec, t->nodes[i], &np);
            }
            if (he != hipSuccess) {
                t->owner = 0;   // nodes partly updated: whoever runs next sets them all
                return he;
            }
            ++g_topo_updated;
        }
    } else {
        if ((int)ts->t.size() >= kTopoPerStream) {
            // replace the least recently used sequence once its last launch has run
            size_t lru = 0;
            for (size_t i = 1; i < ts->t.size(); ++i)
                if (ts->t[i].used < ts->t[lru].used) lru = i;
            Topo& old = ts->t[lru];
            if (old.done) (void)hipEventSynchronize(old.done);
            if (old.exec) (void)hipGraphExecDestroy(old.exec);
            if (old.graph) (void)hipGraphDestroy(old.graph);
            if (old.done) (void)hipEventDestroy(old.done);
            ts->t.erase(ts->t.begin() + lru);
        }
        Topo n;
        n.sig = sig;
        he = hipGraphCreate(&n.graph, 0);
        n.nodes.resize(calls.size());
        for (size_t i = 0; he == hipSuccess && i < calls.size(); ++i) {
            const hipKernelNodeParams np = node_params(calls[i]);
            he = hipGraphAddKernelNode(&n.nodes[i], n.graph, i ? &n.nodes[i - 1] : nullptr, i ? 1 : 0, &np);
        }
        if (he == hipSuccess) he = hipGraphInstantiate(&n.exec, n.graph, nullptr, nullptr, 0);
        if (he == hipSuccess) he = hipEventCreateWithFlags(&n.done, hipEventDisableTiming);
        if (he != hipSuccess) {
            if (n.exec) (void)hipGraphExecDestroy(n.exec);
            if (n.graph) (void)hipGraphDestroy(n.graph);
            return he;
        }
        ++g_topo_instantiated;
        ts->t.push_back(std::move(n));
        t = &ts->t.back();
    }
    t->owner = e->id;
    t->owner_ptrs = ptrs;
    t->used = ++ts->tick;
    he = hipGraphLaunch(t->exec, st);
    if (he == hipSuccess) he = hipEventRecord(t->done, st);
    return he;
}

}  // namespace

namespace {

// Argument checks of an execution (name: the entry point, for the message).
edb_status check_exec_args(const edb_exec* e, const void* const* w, const void* x, const void* arena_h,
                           const void* arena_c, const char* name) {
    const std::string n(name);
    if (!w || !arena_h || !arena_c) return fail(EDB_ERR_INVALID, n + ": NULL argument");
    if (e->n_x > 0 && !x) return fail(EDB_ERR_INVALID, n + ": x is NULL");
    for (int32_t t = 0; t < e->T; ++t)
        if (!w[t]) return fail(EDB_ERR_INVALID, n + ": packed weights of type " + std::to_string(t) + " are NULL");
    auto misaligned = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) != 0; };
    if (misaligned(x) || misaligned(arena_h) || misaligned(arena_c))
        return fail(EDB_ERR_INVALID, n + ": device buffers must be 16-byte aligned");
    for (int32_t t = 0; t < e->T; ++t)
        if (reinterpret_cast<uintptr_t>(w[t]) & 255u)
            return fail(EDB_ERR_INVALID, n + ": packed weights must be 256-byte aligned");
    return EDB_OK;
}

}  // namespace

extern "C" edb_status edb_execute(edb_exec_t* e, const void* const* w, const void* x, void* arena_h,
                                  void* arena_c, void* stream) {
    if (!e) return fail(EDB_ERR_INVALID, "edb_execute: exec is NULL");
    if (e->flags & EDB_DRYRUN) return EDB_OK;
    if (edb_status cs = check_exec_args(e, w, x, arena_h, arena_c, "edb_execute")) return cs;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    hipError_t he = hipStreamWaitEvent(st, e->ready, 0);   // descriptors are on the device
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_execute: ") + hipGetErrorString(he));
    if (!(e->flags & EDB_USE_GRAPH) || (e->flags & EDB_PROFILE)) {
        he = launch_all(e, w, x, arena_h, arena_c, st);
        if (he == hipSuccess) he = hipEventRecord(e->done, st);
        if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_execute: ") + hipGetErrorString(he));
        e->ran = true;
        e->profiled = !e->events.empty();
        return EDB_OK;
    }
    he = graph_launch(e, w, x, arena_h, arena_c, st);
    if (he == hipSuccess) he = hipEventRecord(e->done, st);
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_execute: graph: ") + hipGetErrorString(he));
    e->ran = true;
    return EDB_OK;
}

extern "C" edb_status edb_graph_stats(int64_t* instantiated, int64_t* updated) {
    if (!instantiated || !updated) return fail(EDB_ERR_INVALID, "edb_graph_stats: NULL argument");
    *instantiated = g_topo_instantiated.load();
    *updated = g_topo_updated.load();
    return EDB_OK;
}

namespace {

int64_t align16(int64_t v) { return (v + 15) & ~(int64_t)15; }

// The launch of batch b that holds the batch's own operand lists: its cell
// kernel, or for a child-sum batch on the large tile the child-sum part.
const Launch* batch_launch(const edb_exec* e, int32_t b) {
    for (size_t i = 1; i < e->launches.size(); ++i) {
        const Launch& L = e->launches[i];
        if (!L.flow && L.info.batch == b && L.info.part != 2) return &L;
    }
    return nullptr;
}

// Copy streams of batch b's gather (operand rows -> dense buffer) and scatter
// (dense buffer -> result slots); returns the dense bytes each needs.
void split_streams(const edb_exec* e, const Launch& L, const BatchArgs& a, char* buf, CopyArgs& g, CopyArgs& sc,
                   int64_t& g_bytes, int64_t& s_bytes) {
    const int esz = e->dtype == EDB_F32 ? 4 : 2;
    const int m = a.m, H = a.H;
    g = CopyArgs{};
    sc = CopyArgs{};
    int64_t off = 0;
    auto add = [&](CopyArgs& c, const void* src, Seg srow, int64_t src_rows, void* dst, Seg drow, int64_t dst_rows,
                   int n, int row_bytes) {
        CopyStream& q = c.s[c.n_streams++];
        q.src = reinterpret_cast<const char*>(src);
        q.dst = reinterpret_cast<char*>(dst);
        q.srow = srow;
        q.drow = drow;
        q.n = n;
        q.row_bytes = row_bytes;
        q.src_rows = src_rows;
        q.dst_rows = dst_rows;
    };
    const Seg dense{S_CONTIG, 0, nullptr};
    auto gather = [&](const void* src, Seg srow, int64_t src_rows, int n, int row_bytes) {
        add(g, src, srow, src_rows, buf ? buf + off : nullptr, dense, n, n, row_bytes);
        off = align16(off + (int64_t)n * row_bytes);
    };
    if (a.x.kind != S_NONE && m > 0) gather(a.xmat, a.x, a.n_xrows, m, a.E * esz);
    for (int j = 0; j < 2; ++j)
        if (a.fix[j].kind != S_NONE && m > 0) {
            gather(a.arena_h, a.fix[j], a.n_slots, m, H * esz);
            gather(a.arena_c, a.fix[j], a.n_slots, m, H * 4);
        }
    if (a.rag.kind != S_NONE && L.off_rptr >= 0) {
        const int nrag = e->hbuf[L.off_rptr + m];
        if (nrag > 0) {
            gather(a.arena_h, a.rag, a.n_slots, nrag, H * esz);
            gather(a.arena_c, a.rag, a.n_slots, nrag, H * 4);
        }
    }
    g_bytes = off;
    const int64_t hb = align16((int64_t)m * H * esz);
    if (a.res.kind != S_NONE && m > 0) {
        add(sc, buf, dense, m, a.arena_h, a.res, a.n_slots, m, H * esz);
        add(sc, buf ? buf + hb : nullptr, dense, m, a.arena_c, a.res, a.n_slots, m, H * 4);
    }
    s_bytes = hb + align16((int64_t)m * H * 4);
}

int copy_grid(const CopyArgs& c) {
    int n = 0;
    for (int i = 0; i < c.n_streams; ++i) n = std::max(n, c.s[i].n);
    return (n + 3) / 4;
}

}  // namespace

extern "C" edb_status edb_split_phase_bytes(const edb_exec_t* e, int64_t* bytes) {
    if (!e || !bytes) return fail(EDB_ERR_INVALID, "edb_split_phase_bytes: NULL argument");
    int64_t need = 16;
    for (int32_t b = 0; b < e->B; ++b) {
        const Launch* L = batch_launch(e, b);
        if (!L) return fail(EDB_ERR_UNSUPPORTED, "edb_split_phase_bytes: batch " + std::to_string(b) +
                                                     " runs inside a dataflow launch");
        const BatchArgs a = resolve_args(e, *L, nullptr, nullptr, nullptr, nullptr);
        CopyArgs g, sc;
        int64_t gb = 0, sb = 0;
        split_streams(e, *L, a, nullptr, g, sc, gb, sb);
        need = std::max(need, std::max(gb, sb));
    }
    *bytes = need;
    return EDB_OK;
}

extern "C" edb_status edb_split_phase(edb_exec_t* e, const void* x, void* arena_h, void* arena_c, void* buf,
                                      int64_t buf_bytes, void* stream, float* ms, int32_t n) {
    if (!e) return fail(EDB_ERR_INVALID, "edb_split_phase: exec is NULL");
    if (e->flags & EDB_DRYRUN) return fail(EDB_ERR_INVALID, "edb_split_phase: dry-run executor");
    if (!arena_h || !arena_c || !buf) return fail(EDB_ERR_INVALID, "edb_split_phase: NULL argument");
    if (((e->flags & EDB_X_DIRECT) || e->x_in_place) && e->n_x > 0 && !x)
        return fail(EDB_ERR_INVALID, "edb_split_phase: x is NULL");
    if (!e->ran) return fail(EDB_ERR_INVALID, "edb_split_phase: run edb_execute first (it stages x)");
    if (ms && n < 2 * e->B) return fail(EDB_ERR_INVALID, "edb_split_phase: ms must hold 2 * n_batches values");
    if ((reinterpret_cast<uintptr_t>(buf) | reinterpret_cast<uintptr_t>(arena_h) |
         reinterpret_cast<uintptr_t>(arena_c)) & 15u)
        return fail(EDB_ERR_INVALID, "edb_split_phase: device buffers must be 16-byte aligned");
    int64_t need = 0;
    if (edb_status st = edb_split_phase_bytes(e, &need)) return st;
    if (buf_bytes < need)
        return fail(EDB_ERR_INVALID, "edb_split_phase: buf holds " + std::to_string(buf_bytes) + " bytes, " +
                                         std::to_string(need) + " needed");
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    std::vector<hipEvent_t> ev;
    hipError_t he = hipSuccess;
    if (ms) {
        ev.assign(4 * (size_t)e->B, nullptr);
        for (auto& q : ev)
            if ((he = hipEventCreate(&q)) != hipSuccess) break;
    }
    for (int32_t b = 0; b < e->B && he == hipSuccess; ++b) {
        const Launch* L = batch_launch(e, b);
        const BatchArgs a = resolve_args(e, *L, nullptr, x, arena_h, arena_c);
        CopyArgs g, sc;
        int64_t gb = 0, sb = 0;
        split_streams(e, *L, a, reinterpret_cast<char*>(buf), g, sc, gb, sb);
        const CopyArgs* part[2] = {&g, &sc};
        for (int k = 0; k < 2; ++k) {
            const int gx = copy_grid(*part[k]);
            if (gx > 0 && part[k]->n_streams > 0) {
                const dim3 grid(gx, part[k]->n_streams);
                if (ms)
                    hipExtLaunchKernelGGL(copy_rows_kernel, grid, dim3(256), 0, st, ev[4 * b + 2 * k],
                                          ev[4 * b + 2 * k + 1], 0, *part[k]);
                else
                    hipLaunchKernelGGL(copy_rows_kernel, grid, dim3(256), 0, st, *part[k]);
            } else if (ms) {   // nothing to copy: an empty interval
                he = hipEventRecord(ev[4 * b + 2 * k], st);
                if (he == hipSuccess) he = hipEventRecord(ev[4 * b + 2 * k + 1], st);
            }
            if (he == hipSuccess) he = hipGetLastError();
        }
    }
    if (ms && he == hipSuccess) {
        he = hipStreamSynchronize(st);
        for (int32_t b = 0; b < e->B && he == hipSuccess; ++b)
            for (int k = 0; k < 2 && he == hipSuccess; ++k)
                he = hipEventElapsedTime(&ms[2 * b + k], ev[4 * b + 2 * k], ev[4 * b + 2 * k + 1]);
    }
    for (auto q : ev)
        if (q) (void)hipEventDestroy(q);
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_split_phase: ") + hipGetErrorString(he));
    edb::clear_error();
    return EDB_OK;
}

extern "C" edb_status edb_exec_launches(const edb_exec_t* e, int32_t* n) {
    if (!e || !n) return fail(EDB_ERR_INVALID, "edb_exec_launches: NULL argument");
    *n = (int32_t)e->launches.size();
    return EDB_OK;
}

extern "C" edb_status edb_exec_launch_info(const edb_exec_t* e, int32_t i, edb_launch_info* info) {
    if (!e || !info) return fail(EDB_ERR_INVALID, "edb_exec_launch_info: NULL argument");
    if (i < 0 || i >= (int32_t)e->launches.size()) return fail(EDB_ERR_INVALID, "edb_exec_launch_info: index out of range");
    *info = e->launches[i].info;
    return EDB_OK;
}

extern "C" edb_status edb_exec_launch_times(edb_exec_t* e, float* ms, int32_t n) {
    if (!e || !ms) return fail(EDB_ERR_INVALID, "edb_exec_launch_times: NULL argument");
    if (e->events.empty() || !e->profiled)
        return fail(EDB_ERR_INVALID, "edb_exec_launch_times: no profiled execution");
    if (n != (int32_t)e->launches.size()) return fail(EDB_ERR_INVALID, "edb_exec_launch_times: n != launches");
    hipError_t he = hipEventSynchronize(e->events.back());
    for (int32_t i = 0; he == hipSuccess && i < n; ++i) {
        if (e->launches[i].info.grid == 0) {   // not launched (the staging launch when folded)
            ms[i] = 0.f;
            continue;
        }
        he = hipEventElapsedTime(&ms[i], e->events[2 * i], e->events[2 * i + 1]);
    }
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_exec_launch_times: ") + hipGetErrorString(he));
    return EDB_OK;
}

extern "C" edb_status edb_exec_check(edb_exec_t* e, void* stream) {
    if (!e) return fail(EDB_ERR_INVALID, "edb_exec_check: exec is NULL");
    if ((e->flags & EDB_DRYRUN) || e->n_counters == 0) return EDB_OK;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    hipError_t he = hipStreamSynchronize(st);
    std::vector<int32_t> c((size_t)e->n_counters);
    if (he == hipSuccess)
        he = hipMemcpy(c.data(), e->dbuf + e->off_counters, c.size() * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_exec_check: ") + hipGetErrorString(he));
    for (const Launch& F : e->launches) {
        if (!F.flow) continue;
        if (c[F.f_error - e->off_counters] != 0)
            return fail(EDB_ERR_HIP, "edb_exec_check: a dataflow wait timed out; results are invalid");
    }
    return EDB_OK;
}

extern "C" void edb_exec_free(edb_exec_t* e) { delete e; }

// ---------------------------------------------------------------------------
// edb_forward's plain path.  A call's device memory comes from a block kept
// per device and stream instead of a per-call allocation:
// * its descriptor ints go to one of NH slots, each a device buffer and a
//   pinned host buffer (from a pool kept for the process), used in turn (a
//   copy from pageable memory would be
//   done synchronously, after the copying stream's earlier work): the host
//   fills the pinned buffer; while the stream still runs earlier calls, the
//   device's upload stream copies it, ahead of the stream's kernels, which
//   wait for it (event); on an idle stream a kernel on the stream copies it;
//   a slot is refilled only after the kernels of its last use, NH calls
//   earlier, have finished (event, usually long done);
// * its staged x and scratch rows go to one region, which only kernels on
//   the stream touch, so the next call reuses it in stream order.
// Buffers grow, with a quarter to spare, when a call needs more.  Calls on one
// stream from several threads enqueue one at a time (the block's lock).

namespace {

struct StreamBlock {
    static constexpr int NH = 4;
    struct Slot {
        void* dev = nullptr;        // descriptor ints on the device
        size_t cap = 0;
        void* host = nullptr;       // pinned staging copy
        size_t hcap = 0;
        hipEvent_t ready = nullptr; // the upload has run
        hipEvent_t done = nullptr;  // the kernels that read it have run
        bool used = false;
    };
    std::mutex mu;
    void* rest = nullptr;           // staged x and scratch rows
    size_t rest_cap = 0;
    Slot slot[NH];
    int next = 0;
};
std::mutex g_blocks_mu;
// shared: a release can take a block out of the map while a call still holds it
std::map<std::pair<int, hipStream_t>, std::shared_ptr<StreamBlock>> g_blocks;

// Pinned host memory for the slots, carved from chunks of at least 4 MB that
// are allocated rarely and kept for the process (pinning memory can make the
// runtime wait for the device, which a call inside a busy run must not do).
// A slot that grows takes a new range; the old one is not reused (growth is
// rare, and ranges are a few tens of KB).
struct PinnedPool {
    std::mutex mu;
    uint8_t* cur = nullptr;
    size_t left = 0;
    std::vector<void*> chunks;
};
PinnedPool g_pinned;

hipError_t pinned_range(size_t bytes, void** out) {
    std::lock_guard<std::mutex> lk(g_pinned.mu);
    bytes = (bytes + 255) / 256 * 256;
    if (g_pinned.left < bytes) {
        void* c = nullptr;
        const size_t n = std::max<size_t>(bytes, (size_t)4 << 20);
        // coherent: the upload kernel reads it directly, and a slot's buffer is
        // rewritten every few calls, so the device must not keep old copies
        const hipError_t he = hipHostMalloc(&c, n, hipHostMallocCoherent);
        if (he != hipSuccess) return he;
        g_pinned.chunks.push_back(c);
        g_pinned.cur = reinterpret_cast<uint8_t*>(c);
        g_pinned.left = n;
    }
    *out = g_pinned.cur;
    g_pinned.cur += bytes;
    g_pinned.left -= bytes;
    return hipSuccess;
}

// Descriptor upload by the stream itself: a kernel reads the slot's pinned
// host buffer (the device reads host memory directly) and writes the slot's
// device buffer, 16 bytes a thread.  A copy through the copy engines would
// set up that stream's copy path on its first use (milliseconds, once per
// stream), a kernel runs where the stream's kernels already run.
__global__ __launch_bounds__(256) void upload_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                     int n16) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n16; i += gridDim.x * 256) dst[i] = src[i];
}

// at least one alignment unit, so that no buffer is of zero size
size_t with_spare(size_t v, size_t align) { return std::max(align, (v + v / 4 + align - 1) / align * align); }

}  // namespace

edb_status edb::forward_on_stream(const edb_graph_t* g, const edb_schedule_t* s, const edb_plan_t* p,
                                  const edb_cell* cells, int32_t flags, const void* const* packed_weights,
                                  const void* x, void* arena_h, void* arena_c, void* stream, bool use_graph) {
    int dev = 0;
    DeviceCtx* ctx = nullptr;
    hipError_t he = hipGetDevice(&dev);
    if (he == hipSuccess) he = device_ctx(dev, &ctx);
    if (he == hipSuccess) he = ctx_streams(ctx);
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_forward: ") + hipGetErrorString(he));
    edb_exec_t* e = nullptr;
    edb_status st = prepare_impl(g, s, p, cells, flags, true, &e);
    if (st == EDB_OK) st = check_exec_args(e, packed_weights, x, arena_h, arena_c, "edb_forward");
    std::shared_ptr<StreamBlock> blk;
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    if (st == EDB_OK) {
        std::lock_guard<std::mutex> lk(g_blocks_mu);
        std::shared_ptr<StreamBlock>& up = g_blocks[{dev, hs}];
        if (!up) up.reset(new (std::nothrow) StreamBlock);
        blk = up;
        if (!blk) st = fail(EDB_ERR_OOM, "edb_forward: out of host memory");
    }
    if (st == EDB_OK) {
        std::lock_guard<std::mutex> lk(blk->mu);
        StreamBlock::Slot& sl = blk->slot[blk->next];
        const size_t ibytes = e->d_ibytes, rbytes = e->d_total - e->d_ibytes;
        const size_t hbytes = e->hbuf.size() * sizeof(int32_t);
        // the slot's last kernels have finished: its buffers are free
        if (sl.used) he = hipEventSynchronize(sl.done);
        // Buffers and events: a slot that is too small is resized, and every
        // other slot that is too small and idle with it (never used, or its
        // last kernels finished), so that the next calls on the stream find
        // their slots ready instead of each allocating in turn.  Slot buffers
        // are allocated in the upload stream's order: a call that allocates
        // copies on the upload stream, and the stream's wait for that copy
        // orders it, and every later call on it, after the allocations.
        bool allocated = false;
        for (int k = 0; he == hipSuccess && k < StreamBlock::NH; ++k) {
            StreamBlock::Slot& o = blk->slot[k];
            const bool mine = &o == &sl;
            if (!mine && o.cap >= ibytes && o.hcap >= hbytes && o.ready && o.done) continue;
            if (!mine && o.used) {
                const hipError_t q = hipEventQuery(o.done);
                if (q == hipErrorNotReady) {
                    (void)hipGetLastError();
                    continue;   // still in use: resized when its turn comes
                }
                if (q != hipSuccess) {
                    he = q;
                    break;
                }
            }
            if (!o.ready) he = hipEventCreateWithFlags(&o.ready, hipEventDisableTiming);
            if (he == hipSuccess && !o.done) he = hipEventCreateWithFlags(&o.done, hipEventDisableTiming);
            if (he == hipSuccess && o.cap < ibytes) {
                if (o.dev) (void)hipFreeAsync(o.dev, ctx->upload);
                o.dev = nullptr;
                o.cap = 0;
                const size_t want = with_spare(ibytes, 256);
                he = hipMallocAsync(&o.dev, want, ctx->upload);
                if (he == hipSuccess) o.cap = want;
                else o.dev = nullptr;
                allocated = true;
            }
            if (he == hipSuccess && o.hcap < hbytes) {
                o.host = nullptr;
                o.hcap = 0;
                const size_t want = with_spare(hbytes, 4096);
                he = pinned_range(want, &o.host);
                if (he == hipSuccess) o.hcap = want;
                else o.host = nullptr;
            }
        }
        if (he == hipSuccess && rbytes > 0 && blk->rest_cap < rbytes) {
            // the old region after the stream's earlier kernels
            if (blk->rest) (void)hipFreeAsync(blk->rest, hs);
            blk->rest = nullptr;
            blk->rest_cap = 0;
            const size_t want = with_spare(rbytes, 256);
            he = hipMallocAsync(&blk->rest, want, hs);
            if (he == hipSuccess) blk->rest_cap = want;
            else blk->rest = nullptr;
        }
        // an idle stream (the previous call's kernels have run) copies the
        // descriptors itself: nothing to overlap, and no wait across streams;
        // a busy one has the upload stream copy them ahead of its kernels
        bool idle = !allocated;
        if (he == hipSuccess && idle) {
            const StreamBlock::Slot& prev = blk->slot[(blk->next + StreamBlock::NH - 1) % StreamBlock::NH];
            if (prev.used) {
                const hipError_t q = hipEventQuery(prev.done);
                if (q == hipErrorNotReady) {
                    idle = false;
                    (void)hipGetLastError();
                } else if (q != hipSuccess) {
                    he = q;
                }
            }
        }
        if (he == hipSuccess && hbytes > 0) {
            std::memcpy(sl.host, e->hbuf.data(), hbytes);
            if (idle) {
                // whole 16-byte pieces: both buffers hold at least hbytes
                // rounded up to 256 bytes
                const int n16 = (int)((hbytes + 15) / 16);
                hipLaunchKernelGGL(upload_kernel, dim3(std::min(64, (n16 + 255) / 256)), dim3(256), 0, hs,
                                   reinterpret_cast<const uint4*>(sl.host), reinterpret_cast<uint4*>(sl.dev), n16);
                he = hipGetLastError();
            } else {
                he = hipMemcpyAsync(sl.dev, sl.host, hbytes, hipMemcpyHostToDevice, ctx->upload);
            }
        }
        if (he == hipSuccess && !idle) he = hipEventRecord(sl.ready, ctx->upload);
        if (he == hipSuccess && !idle) he = hipStreamWaitEvent(hs, sl.ready, 0);
        if (he == hipSuccess) {
            // descriptors in the slot; staged x and scratch rows in the region
            // (bound as one block at rest - d_ibytes, whose first d_ibytes are
            // never touched: dbuf is re-pointed to the slot)
            uint8_t* base = blk->rest ? reinterpret_cast<uint8_t*>(blk->rest) - e->d_ibytes
                                      : reinterpret_cast<uint8_t*>(sl.dev);   // no region: no parts past dbuf
            bind_device(e, base);
            e->dbuf = reinterpret_cast<int*>(sl.dev);
            e->dmem = nullptr;
            e->dmem_owned = false;
            he = use_graph ? graph_launch(e, packed_weights, x, arena_h, arena_c, hs)
                           : launch_all(e, packed_weights, x, arena_h, arena_c, hs);
        }
        if (he == hipSuccess) he = hipEventRecord(sl.done, hs);
        if (he == hipSuccess) {
            sl.used = true;
            blk->next = (blk->next + 1) % StreamBlock::NH;
        }
        if (he != hipSuccess) {
            (void)hipGetLastError();
            st = fail(he == hipErrorOutOfMemory ? EDB_ERR_OOM : EDB_ERR_HIP,
                      std::string("edb_forward: ") + hipGetErrorString(he));
        }
    }
    edb_exec_free(e);
    return st;
}

extern "C" edb_status edb_stream_release(void* stream) {
    int dev = 0;
    DeviceCtx* ctx = nullptr;
    hipError_t he = hipGetDevice(&dev);
    if (he == hipSuccess) he = device_ctx(dev, &ctx);
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_stream_release: ") + hipGetErrorString(he));
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    hipError_t ghe = hipSuccess;
    {
        // the stream's kept graphs, each after its last launch (the set itself
        // stays: a graph launch that looked it up before keeps a valid lock)
        TopoSet* ts = nullptr;
        {
            std::lock_guard<std::mutex> lk(g_topo_mu);
            auto it = g_topo.find({dev, hs});
            if (it != g_topo.end()) ts = it->second;
        }
        if (ts) {
            std::lock_guard<std::mutex> lk(ts->mu);
            for (Topo& t : ts->t) {
                if (t.done) {
                    const hipError_t we = hipEventSynchronize(t.done);
                    if (ghe == hipSuccess) ghe = we;
                    (void)hipEventDestroy(t.done);
                }
                if (t.exec) (void)hipGraphExecDestroy(t.exec);
                if (t.graph) (void)hipGraphDestroy(t.graph);
            }
            ts->t.clear();
        }
    }
    std::shared_ptr<StreamBlock> blk;
    {
        std::lock_guard<std::mutex> lk(g_blocks_mu);
        auto it = g_blocks.find({dev, hs});
        if (it == g_blocks.end()) {
            if (ghe != hipSuccess)
                return fail(EDB_ERR_HIP, std::string("edb_stream_release: ") + hipGetErrorString(ghe));
            return EDB_OK;
        }
        blk = std::move(it->second);
        g_blocks.erase(it);
    }
    // a call on the stream that still holds the block finishes enqueueing
    // first (the block's lock); later calls start a new block
    std::lock_guard<std::mutex> lk(blk->mu);
    if (blk->rest) he = hipFreeAsync(blk->rest, hs);
    for (StreamBlock::Slot& sl : blk->slot) {
        // each slot once the kernels of its last use have run
        if (sl.used) {
            const hipError_t we = hipEventSynchronize(sl.done);
            if (he == hipSuccess) he = we;
        }
        if (sl.dev) (void)hipFreeAsync(sl.dev, ctx->upload);
        if (sl.ready) (void)hipEventDestroy(sl.ready);
        if (sl.done) (void)hipEventDestroy(sl.done);
    }
    if (he == hipSuccess) he = ghe;
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_stream_release: ") + hipGetErrorString(he));
    return EDB_OK;
}

// ---------------------------------------------------------------------------
// Allocation-free forward pass: the executor's device memory (descriptor ints,
// staged x, child-sum and MV-RNN scratch rows) lives in one fixed array per
// device instead of a per-call allocation.  Each device that runs this entry
// point holds its own copy of the array for the life of the process; every
// call on a device shares it, so calls that overlap on one device race.

constexpr size_t kNoAllocScratchBytes = (size_t)EDB_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

extern "C" edb_status edb_forward_noalloc(int32_t n_nodes, int32_t n_types, const int32_t* op_type,
                                          const int64_t* child_ptr, const int32_t* child_idx,
                                          const int32_t* x_row, const edb_policy* policy,
                                          const edb_operand_shape* shapes, int32_t plan_flags,
                                          const edb_cell* cells, int32_t exec_flags,
                                          const void* const* packed_weights, const void* x, void* arena_h,
                                          void* arena_c, int64_t arena_rows, void* stream, int32_t* n_slots) {
    if (exec_flags & (EDB_DRYRUN | EDB_PROFILE | EDB_USE_GRAPH))
        return fail(EDB_ERR_INVALID, "edb_forward_noalloc: EDB_DRYRUN, EDB_PROFILE and EDB_USE_GRAPH are not allowed");
    int dev = 0;
    DeviceCtx* ctx = nullptr;
    hipError_t he = hipGetDevice(&dev);
    if (he == hipSuccess) he = device_ctx(dev, &ctx);
    if (he == hipSuccess) {
        // the array's address on this device, looked up once per device (with
        // the device current); the array's name is not a device address in host code
        std::lock_guard<std::mutex> lk(g_ctx_mu);
        if (!ctx->scratch) {
            void* ptr = nullptr;
            he = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
            if (he == hipSuccess) ctx->scratch = ptr;
        }
    }
    if (he != hipSuccess) return fail(EDB_ERR_HIP, std::string("edb_forward_noalloc: ") + hipGetErrorString(he));
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
            st = fail(EDB_ERR_INVALID, "edb_forward_noalloc: the arena has " + std::to_string(arena_rows) +
                                           " rows, the plan needs " + std::to_string(p->n_slots));
    }
    if (st == EDB_OK) st = prepare_impl(g, s, p, cells, exec_flags, true, &e);
    if (st == EDB_OK) st = check_exec_args(e, packed_weights, x, arena_h, arena_c, "edb_forward_noalloc");
    if (st == EDB_OK && e->d_total > kNoAllocScratchBytes)
        st = fail(EDB_ERR_UNSUPPORTED, "edb_forward_noalloc: this mini-batch needs " + std::to_string(e->d_total) +
                                           " bytes of device scratch, the fixed array holds " +
                                           std::to_string(kNoAllocScratchBytes));
    if (st == EDB_OK) {
        bind_device(e, ctx->scratch);
        e->dmem_owned = false;
        hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
        // the descriptors in stream order before the kernels that read them
        // (the host array is read before the call returns: a copy from pageable
        // memory is staged synchronously)
        he = hipMemcpyAsync(e->dbuf, e->hbuf.data(), e->hbuf.size() * sizeof(int32_t), hipMemcpyHostToDevice, hs);
        if (he == hipSuccess) he = launch_all(e, packed_weights, x, arena_h, arena_c, hs);
        if (he != hipSuccess) st = fail(EDB_ERR_HIP, std::string("edb_forward_noalloc: ") + hipGetErrorString(he));
    }
    const std::string err = st == EDB_OK ? std::string() : std::string(edb_last_error());
    edb_exec_free(e);
    edb_plan_free(p);
    edb_schedule_free(s);
    edb_graph_free(g);
    if (st != EDB_OK) return fail(st, err);
    edb::clear_error();
    return EDB_OK;
}

// ---------------------------------------------------------------------------
// Host-side validation of an executor's device descriptors: the int buffer
// that edb_prepare uploads is decoded here the way the kernels read it (the
// same BatchArgs offsets, the same BatchDesc / tile / dependency records of a
// dataflow launch) and every read is bounds-checked; the forward pass is then
// replayed at the level of arena rows (each result slot written once, every
// row read after its producer), and a dataflow launch's ticket and dependency
// protocol is emulated with a bounded number of work-groups.

namespace {

struct VCheck {
    std::string err;
    bool ok() const { return err.empty(); }
    bool fail(const std::string& m) {
        if (err.empty()) err = m;
        return false;
    }
};

// One operand list resolved against the int buffer: entry r's row.
struct VList {
    int kind = S_NONE;
    int base = 0;
    int64_t off = -1;
};

bool v_list(VCheck& c, const std::vector<int32_t>& hb, const VList& l, int64_t n, int64_t rows,
            std::vector<int32_t>& out, const std::string& what) {
    out.clear();
    if (l.kind == S_NONE) return true;
    if (l.kind != S_CONTIG && l.kind != S_INDEXED) return c.fail(what + ": unknown list kind");
    if (n < 0) return c.fail(what + ": negative length");
    if (l.kind == S_INDEXED && (l.off < 0 || l.off + n > (int64_t)hb.size()))
        return c.fail(what + ": index list [" + std::to_string(l.off) + ", +" + std::to_string(n) +
                      ") outside the int buffer of " + std::to_string(hb.size()));
    out.resize((size_t)n);
    for (int64_t r = 0; r < n; ++r) {
        const int64_t v = l.kind == S_CONTIG ? (int64_t)l.base + r : hb[(size_t)(l.off + r)];
        if (v < 0 || v >= rows)
            return c.fail(what + ": entry " + std::to_string(r) + " is row " + std::to_string(v) + " of " +
                          std::to_string(rows));
        out[(size_t)r] = (int32_t)v;
    }
    return true;
}

// The arena rows one batch's cell kernel (or one tile's rows [r0, r1) of it)
// reads and writes, from its lists.
struct VBatch {
    int kind, m, H, Hk, Hu, E, Ep, K, G, nfix;
    bool x, rag;
    VList lx, lf[2], lrag, lres;
    int64_t rptr = -1;
    int64_t n_xrows = 0;
};

bool v_batch_rows(VCheck& c, const std::vector<int32_t>& hb, const VBatch& b, int64_t n_slots, int r0, int r1,
                  std::vector<int32_t>& reads, std::vector<int32_t>& writes, const std::string& what) {
    reads.clear();
    writes.clear();
    std::vector<int32_t> t;
    if (!v_list(c, hb, b.lres, b.m, n_slots, t, what + " result list")) return false;
    if (b.lres.kind != S_NONE)
        for (int r = r0; r < r1; ++r) writes.push_back(t[(size_t)r]);
    for (int p = 0; p < b.nfix; ++p) {
        if (!v_list(c, hb, b.lf[p], b.m, n_slots, t, what + " child list " + std::to_string(p))) return false;
        if (b.lf[p].kind != S_NONE)
            for (int r = r0; r < r1; ++r) reads.push_back(t[(size_t)r]);
    }
    if (b.x && b.lx.kind != S_NONE && !v_list(c, hb, b.lx, b.m, b.n_xrows, t, what + " x list")) return false;
    if (b.rag) {
        if (b.rptr < 0 || b.rptr + b.m + 1 > (int64_t)hb.size())
            return c.fail(what + ": ragged offsets outside the int buffer");
        const int32_t* rp = hb.data() + b.rptr;
        if (rp[0] != 0) return c.fail(what + ": ragged offsets do not start at 0");
        for (int r = 0; r < b.m; ++r)
            if (rp[r + 1] < rp[r]) return c.fail(what + ": ragged offsets decrease at row " + std::to_string(r));
        if (!v_list(c, hb, b.lrag, rp[b.m], n_slots, t, what + " ragged list")) return false;
        if (b.lrag.kind != S_NONE)
            for (int64_t k = rp[r0]; k < rp[r1]; ++k) reads.push_back(t[(size_t)k]);
    }
    // trip counts of the tile loops
    if (b.K <= 0 || b.K > 3 * 4096 + 64) return c.fail(what + ": reduction length " + std::to_string(b.K));
    if (b.Hu % 64 || b.Hu < b.H || b.Hk < b.H) return c.fail(what + ": padded widths");
    return true;
}

}  // namespace

extern "C" edb_status edb_exec_validate(const edb_exec_t* e, int32_t n_workers, int64_t* checked) {
    if (!e) return fail(EDB_ERR_INVALID, "edb_exec_validate: exec is NULL");
    if (n_workers < 1) return fail(EDB_ERR_INVALID, "edb_exec_validate: n_workers must be positive");
    const std::vector<int32_t>& hb = e->hbuf;
    const int64_t n_slots = e->n_slots;
    const bool x_caller = (e->flags & EDB_X_DIRECT) || e->x_in_place;
    const int64_t n_xrows = x_caller ? e->x_direct_rows : e->n_x;
    VCheck c;
    int64_t n_checked = 0;
    // rows: -2 never written, -1 zero / pad row (cleared before any batch), else the writing launch
    std::vector<int64_t> written((size_t)n_slots, -2);
    // the zero row and the pads
    if (e->off_zero < 0 || e->off_zero + e->n_zero > (int64_t)hb.size())
        return fail(EDB_ERR_INVALID, "edb_exec_validate: zero-row list outside the int buffer");
    for (int i = 0; i < e->n_zero; ++i) {
        const int64_t z = hb[(size_t)(e->off_zero + i)];
        if (z < 0 || z >= n_slots) return fail(EDB_ERR_INVALID, "edb_exec_validate: zero/pad row out of range");
        written[(size_t)z] = -1;
    }
    if (hb[(size_t)e->off_zero] != 0) return fail(EDB_ERR_INVALID, "edb_exec_validate: the zero row is not slot 0");
    // staged x source rows
    if (!x_caller && e->n_x > 0) {
        if (e->off_xsrc < 0 || e->off_xsrc + e->n_x > (int64_t)hb.size())
            return fail(EDB_ERR_INVALID, "edb_exec_validate: x source rows outside the int buffer");
        for (int32_t i = 0; i < e->n_x; ++i) {
            const int32_t r = hb[(size_t)(e->off_xsrc + i)];
            if (r < 0 || r >= e->x_direct_rows)
                return fail(EDB_ERR_INVALID, "edb_exec_validate: x source row " + std::to_string(r) + " out of range");
        }
    }
    // the dataflow counters are zero in the upload and the staging launch clears them
    if (e->off_counters < 0 || e->off_counters + e->n_counters > (int64_t)hb.size())
        return fail(EDB_ERR_INVALID, "edb_exec_validate: counter region outside the int buffer");
    for (int64_t i = 0; i < e->n_counters; ++i)
        if (hb[(size_t)(e->off_counters + i)] != 0) return fail(EDB_ERR_INVALID, "edb_exec_validate: counter not zero");
    if (e->n_counters > 0 && e->launches[0].info.grid == 0)
        return fail(EDB_ERR_INVALID, "edb_exec_validate: dataflow counters but no staging launch to clear them");

    auto batch_of = [&](const Launch& L) {
        VBatch b{};
        const Dims& d = e->dims[L.type];
        const KindInfo ki = kind_info(e->cells[L.type].kind);
        b.kind = L.info.kind;
        b.m = L.args.m;
        b.H = d.H; b.Hk = d.Hk; b.Hu = d.Hu; b.E = d.E; b.Ep = d.Ep; b.K = d.K; b.G = d.G;
        b.nfix = ki.nfix;
        b.x = ki.x;
        b.rag = ki.rag;
        b.lx = VList{L.args.x.kind, L.args.x.base, L.off_x};
        b.lf[0] = VList{L.args.fix[0].kind, L.args.fix[0].base, L.off_f0};
        b.lf[1] = VList{L.args.fix[1].kind, L.args.fix[1].base, L.off_f1};
        b.lrag = VList{L.args.rag.kind, L.args.rag.base, L.off_rag};
        b.lres = VList{L.args.res.kind, L.args.res.base, L.off_res};
        b.rptr = L.off_rptr;
        b.n_xrows = n_xrows;
        return b;
    };
    std::vector<int32_t> rd, wr;
    auto commit = [&](int64_t li, const std::string& what) {
        for (int32_t v : rd)
            if (written[(size_t)v] == -2)
                return c.fail(what + ": reads row " + std::to_string(v) + " before any launch writes it");
        for (int32_t v : wr) {
            if (v == 0 || written[(size_t)v] == -1)
                return c.fail(what + ": writes the zero row or a pad row (" + std::to_string(v) + ")");
            if (written[(size_t)v] != -2)
                return c.fail(what + ": writes row " + std::to_string(v) + " a second time");
            written[(size_t)v] = li;
        }
        return true;
    };

    for (size_t li = 1; li < e->launches.size() && c.ok(); ++li) {
        const Launch& L = e->launches[li];
        const std::string what = "launch " + std::to_string(li) + " (batch " + std::to_string(L.info.batch) + ")";
        if (!L.flow) {
            if (L.kk < 0 || L.info.part != 0) {
                // the parts before a batch's cell kernel read its lists; they write scratch rows only
                VBatch b = batch_of(L);
                b.lres.kind = S_NONE;
                if (L.info.part == 2) {   // forget GEMM: x = the child list, m = children
                    b.rag = false;
                    b.nfix = 0;
                    b.x = true;
                    b.lx = VList{L.args.x.kind, L.args.x.base, L.off_x};
                    b.n_xrows = n_slots;
                    std::vector<int32_t> t;
                    if (!v_list(c, hb, b.lx, L.args.m, n_slots, t, what + " child rows")) break;
                    for (int32_t v : t)
                        if (written[(size_t)v] == -2) { c.fail(what + ": reads an unwritten child row"); break; }
                    ++n_checked;
                    continue;
                }
                b.x = false;
                if (!v_batch_rows(c, hb, b, n_slots, 0, b.m, rd, wr, what)) break;
                wr.clear();
                if (!commit((int64_t)li, what)) break;
                ++n_checked;
                continue;
            }
            VBatch b = batch_of(L);
            if (b.lres.kind == S_NONE) { c.fail(what + ": no result list"); break; }
            if (L.kk == K_CS_PARENT || L.kk == K_MV_VEC) b.x = false;   // rows from scratch written just before
            if (L.kk == K_CS_PARENT) b.rag = false;                     // its children were read by the parts
            if (!v_batch_rows(c, hb, b, n_slots, 0, b.m, rd, wr, what)) break;
            if (!commit((int64_t)li, what)) break;
            ++n_checked;
            continue;
        }
        // ---- dataflow launch ----
        const int nb = L.info.n_batches;
        if (L.f_desc < 0 || L.f_desc % 4 || L.f_desc + (int64_t)nb * (int64_t)(sizeof(BatchDesc) / 4) > (int64_t)hb.size())
            { c.fail(what + ": batch descriptors outside the int buffer or misaligned"); break; }
        const BatchDesc* bd = reinterpret_cast<const BatchDesc*>(hb.data() + L.f_desc);
        const int need = L.f_need;
        std::vector<VBatch> vb((size_t)nb);
        std::vector<int> rt_base((size_t)nb + 1, 0);
        for (int q = 0; q < nb && c.ok(); ++q) {
            const BatchDesc& d = bd[q];
            if (d.type < 0 || d.type >= e->T) { c.fail(what + ": descriptor type"); break; }
            const KindInfo ki = kind_info(d.kind);
            if (ki.G == 0 || d.kind != e->cells[d.type].kind) { c.fail(what + ": descriptor kind"); break; }
            const Dims& dm = e->dims[d.type];
            if (d.H != dm.H || d.Hk != dm.Hk || d.Hu != dm.Hu || d.E != dm.E || d.Ep != dm.Ep || d.K != dm.K)
                { c.fail(what + ": descriptor dimensions differ from the cell's"); break; }
            if (d.off_b != (int)dm.off_b || d.off_Wr != (int)dm.off_Wr || d.off_br != (int)dm.off_br)
                { c.fail(what + ": descriptor weight offsets"); break; }
            if (d.x_staged != (x_caller ? 0 : 1)) { c.fail(what + ": descriptor x source"); break; }
            if (d.m < 1) { c.fail(what + ": empty batch in a run"); break; }
            VBatch& b = vb[(size_t)q];
            b.kind = d.kind; b.m = d.m; b.H = d.H; b.Hk = d.Hk; b.Hu = d.Hu; b.E = d.E; b.Ep = d.Ep; b.K = d.K;
            b.G = ki.G; b.nfix = ki.nfix; b.x = ki.x; b.rag = ki.rag;
            VList* ls[5] = {&b.lx, &b.lf[0], &b.lf[1], &b.lrag, &b.lres};
            for (int i = 0; i < 5; ++i) *ls[i] = VList{d.seg_kind[i], d.seg_base[i], d.seg_off[i]};
            b.rptr = d.rptr_off;
            b.n_xrows = n_xrows;
            if (b.Hu / (16 * FLOW_WU) != need) { c.fail(what + ": unit tiles of a batch differ from `need`"); break; }
            rt_base[(size_t)q + 1] = rt_base[(size_t)q] + (d.m + 16 * FLOW_RT - 1) / (16 * FLOW_RT);
        }
        if (!c.ok()) break;
        const int nrt = rt_base[(size_t)nb];
        if (L.f_tiles < 0 || L.f_tiles % 4 || L.f_tiles + 4LL * L.f_ntiles > (int64_t)hb.size())
            { c.fail(what + ": tile records outside the int buffer or misaligned"); break; }
        if (L.f_rtdeps < 0 || L.f_rtdeps % 2 || L.f_rtdeps + 2LL * nrt > (int64_t)hb.size())
            { c.fail(what + ": dependency ranges outside the int buffer or misaligned"); break; }
        if (L.f_ticket < e->off_counters || L.f_error != L.f_ticket + 1 || L.f_done != L.f_ticket + 2 ||
            L.f_done + nrt > e->off_counters + e->n_counters)
            { c.fail(what + ": counters outside the counter region"); break; }
        if (L.args.m < 1) { c.fail(what + ": wait bound"); break; }
        if (L.info.grid < 1 || L.info.grid > L.f_ntiles) { c.fail(what + ": grid"); break; }
        const int4* tiles = reinterpret_cast<const int4*>(hb.data() + L.f_tiles);
        const int2* rdep = reinterpret_cast<const int2*>(hb.data() + L.f_rtdeps);
        // tiles in (batch, row tile, unit tile) order, `need` unit tiles per row tile
        std::vector<int> first_ticket((size_t)nrt, -1), last_ticket((size_t)nrt, -1), count((size_t)nrt, 0);
        std::vector<int> rt_batch((size_t)nrt, -1), rt_row((size_t)nrt, -1);
        for (int t = 0; t < L.f_ntiles && c.ok(); ++t) {
            const int4 tl = tiles[t];
            if (tl.x < 0 || tl.x >= nb) { c.fail(what + ": tile " + std::to_string(t) + " batch"); break; }
            const VBatch& b = vb[(size_t)tl.x];
            if (tl.y < 0 || tl.y * 16 * FLOW_RT >= b.m) { c.fail(what + ": tile " + std::to_string(t) + " row tile"); break; }
            if (tl.z < 0 || tl.z >= need) { c.fail(what + ": tile " + std::to_string(t) + " unit tile"); break; }
            if (tl.w != rt_base[(size_t)tl.x] + tl.y) { c.fail(what + ": tile " + std::to_string(t) + " row-tile id"); break; }
            if (t > 0) {
                const int4 p = tiles[t - 1];
                if (std::make_tuple(p.x, p.y, p.z) >= std::make_tuple(tl.x, tl.y, tl.z))
                    { c.fail(what + ": tiles out of order at " + std::to_string(t)); break; }
            }
            if (first_ticket[(size_t)tl.w] < 0) first_ticket[(size_t)tl.w] = t;
            last_ticket[(size_t)tl.w] = t;
            ++count[(size_t)tl.w];
            rt_batch[(size_t)tl.w] = tl.x;
            rt_row[(size_t)tl.w] = tl.y;
        }
        if (!c.ok()) break;
        for (int r = 0; r < nrt; ++r)
            if (count[(size_t)r] != need) { c.fail(what + ": row tile " + std::to_string(r) + " has " +
                                                   std::to_string(count[(size_t)r]) + " unit tiles, need " +
                                                   std::to_string(need)); break; }
        if (!c.ok()) break;
        int64_t ndeps = 0;
        for (int r = 0; r < nrt; ++r) ndeps = std::max<int64_t>(ndeps, (int64_t)rdep[r].x + rdep[r].y);
        if (L.f_deps < 0 || L.f_deps + ndeps > (int64_t)hb.size()) { c.fail(what + ": dependency list outside"); break; }
        const int32_t* deps = hb.data() + L.f_deps;
        // per row tile: its reads are produced by earlier launches or by its
        // dependencies, whose every unit tile holds a smaller ticket
        std::vector<int64_t> run_writer((size_t)n_slots, -1);   // row tile of this run writing the slot
        for (int q = 0; q < nb; ++q)
            if (vb[(size_t)q].lres.kind == S_NONE) c.fail(what + ": batch " + std::to_string(q) + " has no result list");
        for (int r = 0; r < nrt && c.ok(); ++r) {
            const VBatch& b = vb[(size_t)rt_batch[(size_t)r]];
            const int r0 = rt_row[(size_t)r] * 16 * FLOW_RT, r1 = std::min(b.m, r0 + 16 * FLOW_RT);
            const std::string tw = what + " row tile " + std::to_string(r);
            if (!v_batch_rows(c, hb, b, n_slots, r0, r1, rd, wr, tw)) break;
            const int2 di = rdep[r];
            if (di.x < 0 || di.y < 0) { c.fail(tw + ": dependency range"); break; }
            std::vector<int> dl(deps + di.x, deps + di.x + di.y);
            for (int dp : dl) {
                if (dp < 0 || dp >= nrt) { c.fail(tw + ": dependency " + std::to_string(dp) + " out of range"); break; }
                if (last_ticket[(size_t)dp] >= first_ticket[(size_t)r])
                    { c.fail(tw + ": depends on row tile " + std::to_string(dp) + " with a later ticket"); break; }
            }
            if (!c.ok()) break;
            for (int32_t v : rd) {
                if (written[(size_t)v] != -2) continue;   // zero / pad row or an earlier launch
                const int64_t pw = run_writer[(size_t)v];
                if (pw < 0) { c.fail(tw + ": reads row " + std::to_string(v) + " that nothing before it writes"); break; }
                if (std::find(dl.begin(), dl.end(), (int)pw) == dl.end())
                    { c.fail(tw + ": reads row " + std::to_string(v) + " of row tile " + std::to_string(pw) +
                             ", which is not among its dependencies"); break; }
            }
            for (int32_t v : wr) {
                if (v == 0 || written[(size_t)v] != -2 || run_writer[(size_t)v] >= 0)
                    { c.fail(tw + ": writes row " + std::to_string(v) + " that is written elsewhere"); break; }
                run_writer[(size_t)v] = r;
            }
            ++n_checked;
        }
        if (!c.ok()) break;
        for (int64_t v = 0; v < n_slots; ++v)
            if (run_writer[(size_t)v] >= 0) written[(size_t)v] = (int64_t)li;
        // the ticket protocol with W work-groups, several interleavings: each
        // work-group claims the next ticket when idle, waits until every unit
        // tile of each dependency has finished, finishes its tile a step later
        const int W = std::max(1, std::min<int>(n_workers, L.info.grid));
        for (uint64_t seed = 1; seed <= 4 && c.ok(); ++seed) {
            std::vector<int> done_ctr((size_t)nrt, 0), hold((size_t)W, -1);
            int ticket = 0, finished = 0;
            uint64_t rng = seed * 0x9E3779B97F4A7C15ull;
            int64_t idle_rounds = 0;
            while (finished < L.f_ntiles) {
                bool progress = false;
                for (int k = 0; k < W; ++k) {
                    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
                    const int wgi = (int)(rng % (uint64_t)W);
                    int& h = hold[(size_t)wgi];
                    if (h < 0) {
                        if (ticket < L.f_ntiles) { h = ticket++; progress = true; }
                        continue;
                    }
                    const int r = tiles[h].w;
                    bool ready = true;
                    for (int i = 0; i < rdep[r].y; ++i)
                        if (done_ctr[(size_t)deps[rdep[r].x + i]] < need) { ready = false; break; }
                    if (ready) {
                        ++done_ctr[(size_t)r];
                        ++finished;
                        h = -1;
                        progress = true;
                    }
                }
                idle_rounds = progress ? 0 : idle_rounds + 1;
                if (idle_rounds > 4LL * W + 16) {
                    c.fail(what + ": the ticket protocol does not drain with " + std::to_string(W) +
                           " work-groups (" + std::to_string(finished) + " of " + std::to_string(L.f_ntiles) +
                           " tiles finished)");
                    break;
                }
            }
        }
    }
    if (c.ok())
        for (int64_t v = 0; v < n_slots; ++v)
            if (written[(size_t)v] == -2) {
                // a slot that no launch writes and that is not a zero / pad row
                c.fail("slot " + std::to_string(v) + " is never written");
                break;
            }
    if (checked) *checked = n_checked;
    if (!c.ok()) return fail(EDB_ERR_INVALID, "edb_exec_validate: " + c.err);
    edb::clear_error();
    return EDB_OK;
}
