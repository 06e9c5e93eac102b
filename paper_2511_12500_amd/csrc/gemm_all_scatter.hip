// One rank's share of GEMM + All-Scatter (Section 4 of the paper), on gfx950.
//
// Problem (Section 4, case study): rank r holds A [M, K] and the column
// shard B_r [K, N] (N = N_local) of a column-parallel GEMM.  It computes
// C_r = A * B_r and makes it the column block [r*N, (r+1)*N) of the
// gathered output [M, w*N] in every rank's heap.
//
// Kernel structure (this file's design, not the paper's Triton code):
//   * persistent grid; producer workgroup g takes tiles g, g+G, g+2G, ...
//     (the persistent tile loop of Sections 4.1.1 and 4.2.1);
//   * tile -> (tile row, tile column): an XCD-aware remap (workgroups are
//     dispatched round-robin over the 8 XCDs, so the tiles in flight on one
//     XCD are made spatial neighbours) followed by a GROUP_M swizzle
//     (Section 3.4, swizzling);
//   * main loop (Section 4, GEMM main-loop listing): 4 waves in a 2 x 2
//     layout, each owning a (BM/2) x (BN/2) block of 32x32 MFMA
//     accumulators (v_mfma_f32_32x32x16_{bf16,f16}, fp32 accumulate);
//     A and B tiles of BK = 64 are staged through LDS, double buffered, with
//     an XOR swizzle that keeps both the staging writes and the fragment
//     reads free of bank conflicts;  B arrives row-major (N contiguous) and
//     is transposed 8x8 in registers while staging, so every MFMA operand
//     is a single 16-byte LDS read of 8 consecutive k;
//   * epilogue (Section 4.2.1): the accumulators are rounded to the output
//     type (nearest even), restaged through LDS as row-major 16-byte
//     chunks and written with coalesced 128-bit stores to each destination
//     heap (value-based store through the translated address), then the
//     per-tile counters are released at agent scope.
//   * workgroup specialisation (Section 4.2.2): with variant WG_SPEC the
//     first gemm_wgs workgroups produce into the local heap and release a
//     per-tile ready counter; the remaining copy_wgs workgroups acquire it
//     and put the tile into the other w-1 heaps (pointer-based put).
//   * bulk-synchronous (Section 4.1.1): producers store locally, and a
//     second kernel on the same stream puts every tile to the other heaps.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "symtile.h"
#include "symtile_device.h"
#include "symtile_internal.h"

namespace {

using symtile::u32x4;
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int BK = 64;                 // K depth of one staged tile
constexpr int kRowBytes = BK * 2;      // LDS bytes per staged row (8 chunks of 16 B)

enum KernelRole : int { ROLE_LOCAL_ONLY = 0, ROLE_FUSED = 1, ROLE_WG_SPEC = 2 };

struct GasParams {
    const uint16_t* A;
    const uint16_t* B;
    uint16_t* C;            // gathered output, column 0, in slot `rank`
    uint32_t* arrived;      // [world][tiles_m][tiles_n] in slot `rank`
    uint32_t* ready;        // [tiles_m * tiles_n], WG_SPEC only
    const uint64_t* bases;
    uint32_t* err;
    int M, N, K;
    int lda, ldb, ldc;
    int rank, world;
    int tiles_m, tiles_n, num_tiles;
    int role;
    int gemm_wgs, copy_wgs;
    int group_m;
    uint32_t epoch, spin_limit;
    int nontemporal;
};

// XOR swizzle of the 16-byte chunk index inside a 128-byte staged row.
__device__ __forceinline__ int swz(int row) { return (row ^ (row >> 3)) & 7; }

// Producer-order tile index t -> (tile row, tile column).
__device__ __forceinline__ void tile_coords(int t, int G, const GasParams& p, int& tm, int& tn) {
    int L = t;
    const int round = t / G;
    if ((G & 7) == 0 && (round + 1) * G <= p.num_tiles) {
        const int pos = t - round * G;
        L = round * G + (pos & 7) * (G >> 3) + (pos >> 3);
    }
    const int width = p.group_m * p.tiles_n;
    const int group = L / width;
    const int first_m = group * p.group_m;
    const int gsize = min(p.tiles_m - first_m, p.group_m);
    const int in = L - group * width;
    tm = first_m + in % gsize;
    tn = in / gsize;
}

template <bool BF16>
__device__ __forceinline__ f32x16_t mfma32(u32x4 a, u32x4 b, f32x16_t c) {
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                       __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                      __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// Round two fp32 values to the 16-bit output type (nearest even) and pack.
template <bool BF16>
__device__ __forceinline__ uint32_t cvt_pack(float x, float y) {
    uint16_t a, b;
    if constexpr (BF16) {
        a = __builtin_bit_cast(uint16_t, (__bf16)x);
        b = __builtin_bit_cast(uint16_t, (__bf16)y);
    } else {
        a = __builtin_bit_cast(uint16_t, (_Float16)x);
        b = __builtin_bit_cast(uint16_t, (_Float16)y);
    }
    return (uint32_t)a | ((uint32_t)b << 16);
}

// ---------------------------------------------------------------------------
// Copy one finished tile from the local heap to every other heap (the put of
// Sections 4.1.1 and 4.2.2) and release its counters there.
template <int BM, int BN>
__device__ void put_tile_to_peers(const GasParams& p, int tm, int tn) {
    constexpr int CPR = BN / 8;                 // 16-byte chunks per tile row
    constexpr int TOTAL = BM * CPR;
    constexpr int PER = TOTAL / kThreads;
    constexpr int U = PER < 8 ? PER : 8;
    static_assert(TOTAL % kThreads == 0, "tile must split evenly over the threads");
    const int m0 = tm * BM, n0 = tn * BN;
    const uint16_t* src = p.C + (size_t)p.rank * p.N;
    const bool nt = p.nontemporal != 0;
#pragma unroll 1
    for (int b = 0; b < PER; b += U) {
        u32x4 v[U];
        size_t off[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int q = threadIdx.x + (b + u) * kThreads;
            const int row = q / CPR, c = q % CPR;
            ok[u] = (m0 + row < p.M) && (n0 + 8 * c < p.N);
            off[u] = (size_t)(m0 + row) * p.ldc + (size_t)(n0 + 8 * c);
            if (ok[u]) v[u] = symtile::ld16(src + off[u]);
        }
        for (int d = 1; d < p.world; ++d) {
            const int s = (p.rank + d) % p.world;
            uint16_t* dst = symtile::translate(const_cast<uint16_t*>(src), p.rank, s, p.bases);
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (ok[u]) symtile::st16(dst + off[u], v[u], nt);
        }
    }
    symtile::wg_release_begin();
    if (threadIdx.x == 0) {
        uint32_t* flag = p.arrived + ((size_t)p.rank * p.tiles_m + tm) * p.tiles_n + tn;
        for (int d = 1; d < p.world; ++d)
            symtile::flag_add_release(
                symtile::translate(flag, p.rank, (p.rank + d) % p.world, p.bases));
    }
}

// ---------------------------------------------------------------------------
template <int BM, int BN, bool BF16>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gas_kernel(const GasParams p) {
    constexpr int WM = BM / 2, WN = BN / 2;     // wave tile
    constexpr int MI = WM / 32, NI = WN / 32;   // 32x32 MFMA blocks per wave
    constexpr int A_BYTES = BM * kRowBytes, B_BYTES = BN * kRowBytes;
    constexpr int STAGE = A_BYTES + B_BYTES;
    constexpr int C_BYTES = BM * BN * 2;
    constexpr int LDS_BYTES = (2 * STAGE > C_BYTES) ? 2 * STAGE : C_BYTES;
    constexpr int A_LD = BM * (BK / 8) / kThreads;      // A chunks per thread
    constexpr int B_UNITS = (BN / 8) * (BK / 8);        // (n chunk, 8-row k group) pairs
    constexpr int B_LD = (B_UNITS + kThreads - 1) / kThreads;
    static_assert(MI >= 1 && NI >= 1 && WM % 32 == 0 && WN % 32 == 0, "unsupported tile");
    static_assert(BM * (BK / 8) % kThreads == 0, "A tile must split evenly");

    __shared__ __attribute__((aligned(16))) uint8_t smem[LDS_BYTES];
    __shared__ int s_ok;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int pid = blockIdx.x;

    // ---------------- consumer workgroups (Section 4.2.2) -----------------
    if (p.role == ROLE_WG_SPEC && pid >= p.gemm_wgs) {
        const int cid = pid - p.gemm_wgs;
        for (int t = cid; t < p.num_tiles; t += p.copy_wgs) {
            int tm, tn;
            tile_coords(t, p.gemm_wgs, p, tm, tn);
            if (tid == 0) {
                const bool ok =
                    symtile::flag_wait_geq(p.ready + tm * p.tiles_n + tn, p.epoch, p.spin_limit);
                if (ok)
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                else
                    symtile::raise_error(p.err, symtile::ERR_TIMEOUT);
                s_ok = ok;
            }
            __syncthreads();
            if (!s_ok) return;
            put_tile_to_peers<BM, BN>(p, tm, tn);
        }
        return;
    }

    // ---------------- producer workgroups ---------------------------------
    const int G = p.gemm_wgs;
    const int KT = (p.K + BK - 1) / BK;
    const bool nt = p.nontemporal != 0;

    for (int t = pid; t < p.num_tiles; t += G) {
        int tm, tn;
        tile_coords(t, G, p, tm, tn);
        const int m0 = tm * BM, n0 = tn * BN;

        f32x16_t acc[MI][NI];
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NI; ++j)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

        u32x4 ra[A_LD];
        u32x4 rb[B_LD][8];

        // Global -> registers for K tile kt (zero outside the matrices).
        auto load_tile = [&](int kt) {
            const int k0 = kt * BK;
#pragma unroll
            for (int u = 0; u < A_LD; ++u) {
                const int q = tid + u * kThreads;
                const int row = q >> 3, c = q & 7;
                const int gr = m0 + row, gk = k0 + 8 * c;
                ra[u] = (gr < p.M && gk < p.K)
                            ? symtile::ld16(p.A + (size_t)gr * p.lda + gk)
                            : u32x4{0, 0, 0, 0};
            }
#pragma unroll
            for (int u = 0; u < B_LD; ++u) {
                const int v = tid + u * kThreads;
                const int nc = v % (BN / 8), kg = v / (BN / 8);
                const int gn = n0 + 8 * nc;
                const bool col_ok = v < B_UNITS && gn < p.N;
#pragma unroll
                for (int r = 0; r < 8; ++r) {
                    const int gk = k0 + 8 * kg + r;
                    rb[u][r] = (col_ok && gk < p.K)
                                   ? symtile::ld16(p.B + (size_t)gk * p.ldb + gn)
                                   : u32x4{0, 0, 0, 0};
                }
            }
        };

        // Registers -> LDS stage `buf`; B is transposed 8x8 on the way so
        // that each staged B row holds 8 consecutive k of one column.
        auto stage_tile = [&](int buf) {
            uint8_t* As = smem + buf * STAGE;
            uint8_t* Bs = As + A_BYTES;
#pragma unroll
            for (int u = 0; u < A_LD; ++u) {
                const int q = tid + u * kThreads;
                const int row = q >> 3, c = q & 7;
                *reinterpret_cast<u32x4*>(As + row * kRowBytes + ((c ^ swz(row)) << 4)) = ra[u];
            }
#pragma unroll
            for (int u = 0; u < B_LD; ++u) {
                const int v = tid + u * kThreads;
                if (v < B_UNITS) {
                    const int nc = v % (BN / 8), kg = v / (BN / 8);
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int d = j >> 1;
                        u32x4 col;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const uint32_t x = rb[u][2 * e][d], y = rb[u][2 * e + 1][d];
                            col[e] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u))
                                             : ((x & 0xFFFFu) | (y << 16));
                        }
                        const int n = nc * 8 + j;
                        *reinterpret_cast<u32x4*>(Bs + n * kRowBytes + ((kg ^ swz(n)) << 4)) = col;
                    }
                }
            }
        };

        // MFMAs over LDS stage `buf`.  Operands are swapped (B fragment as
        // the first source) so each lane's accumulators hold 4 consecutive
        // columns of one row of C, which makes the epilogue restage cheap.
        auto compute_tile = [&](int buf) {
            const uint8_t* As = smem + buf * STAGE;
            const uint8_t* Bs = As + A_BYTES;
#pragma unroll
            for (int s = 0; s < BK / 16; ++s) {
                const int c = 2 * s + (lane >> 5);
                u32x4 a[MI], b[NI];
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int row = wm * WM + i * 32 + (lane & 31);
                    a[i] = *reinterpret_cast<const u32x4*>(As + row * kRowBytes +
                                                          ((c ^ swz(row)) << 4));
                }
#pragma unroll
                for (int j = 0; j < NI; ++j) {
                    const int row = wn * WN + j * 32 + (lane & 31);
                    b[j] = *reinterpret_cast<const u32x4*>(Bs + row * kRowBytes +
                                                          ((c ^ swz(row)) << 4));
                }
#pragma unroll
                for (int i = 0; i < MI; ++i)
#pragma unroll
                    for (int j = 0; j < NI; ++j) acc[i][j] = mfma32<BF16>(b[j], a[i], acc[i][j]);
            }
        };

        if (KT > 0) {
            load_tile(0);
            stage_tile(0);
            __syncthreads();
        }
        for (int kt = 0; kt < KT; ++kt) {
            const int cur = kt & 1;
            if (kt + 1 < KT) load_tile(kt + 1);
            compute_tile(cur);
            if (kt + 1 < KT) stage_tile(cur ^ 1);
            __syncthreads();
        }

        // ---- epilogue: round, restage row-major, store, release --------
        uint8_t* Cs = smem;
        constexpr int CROW = BN * 2;               // bytes per staged C row
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NI; ++j)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int row = wm * WM + i * 32 + (lane & 31);
                    const int col = wn * WN + j * 32 + 8 * g + 4 * (lane >> 5);
                    uint2 w;
                    w.x = cvt_pack<BF16>(acc[i][j][4 * g + 0], acc[i][j][4 * g + 1]);
                    w.y = cvt_pack<BF16>(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                    const int chunk = col >> 3, half = (col >> 2) & 1;
                    *reinterpret_cast<uint2*>(Cs + row * CROW + ((chunk ^ (row & 7)) << 4) +
                                              (half << 3)) = w;
                }
        __syncthreads();

        const int n_dst = (p.role == ROLE_FUSED) ? p.world : 1;
        uint16_t* cbase = p.C + (size_t)p.rank * p.N;
        {
            constexpr int CPR = BN / 8;
            constexpr int TOTAL = BM * CPR;
            constexpr int PER = TOTAL / kThreads;
            constexpr int U = PER < 8 ? PER : 8;
            static_assert(TOTAL % kThreads == 0, "tile must split evenly over the threads");
#pragma unroll 1
            for (int b = 0; b < PER; b += U) {
                u32x4 v[U];
                size_t off[U];
                bool ok[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int q = tid + (b + u) * kThreads;
                    const int row = q / CPR, c = q % CPR;
                    v[u] = *reinterpret_cast<const u32x4*>(Cs + row * CROW +
                                                          ((c ^ (row & 7)) << 4));
                    ok[u] = (m0 + row < p.M) && (n0 + 8 * c < p.N);
                    off[u] = (size_t)(m0 + row) * p.ldc + (size_t)(n0 + 8 * c);
                }
                for (int d = 0; d < n_dst; ++d) {
                    const int s = (p.rank + d) % p.world;
                    uint16_t* dst = symtile::translate(cbase, p.rank, s, p.bases);
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        if (ok[u]) symtile::st16(dst + off[u], v[u], nt);
                }
            }
        }
        symtile::wg_release_begin();   // also orders the LDS reads above before reuse
        if (tid == 0) {
            uint32_t* flag = p.arrived + ((size_t)p.rank * p.tiles_m + tm) * p.tiles_n + tn;
            for (int d = 0; d < n_dst; ++d)
                symtile::flag_add_release(
                    symtile::translate(flag, p.rank, (p.rank + d) % p.world, p.bases));
            if (p.role == ROLE_WG_SPEC) symtile::flag_add_release(p.ready + tm * p.tiles_n + tn);
        }
    }
}

// Second kernel of the bulk-synchronous schedule (Section 4.1.1).
template <int BM, int BN>
__global__ __launch_bounds__(kThreads) void scatter_kernel(const GasParams p) {
    for (int t = blockIdx.x; t < p.num_tiles; t += gridDim.x) {
        const int tm = t / p.tiles_n, tn = t % p.tiles_n;
        put_tile_to_peers<BM, BN>(p, tm, tn);
    }
}

// ---------------------------------------------------------------------------
struct Variant {
    int bm, bn;
    bool bf16;
    const void* gas;
    const void* scatter;
};

template <int BM, int BN, bool BF16>
Variant make_variant() {
    return Variant{BM, BN, BF16, reinterpret_cast<const void*>(&gas_kernel<BM, BN, BF16>),
                   reinterpret_cast<const void*>(&scatter_kernel<BM, BN>)};
}

const Variant* find_variant(int bm, int bn, bool bf16) {
    static const Variant table[] = {
        make_variant<64, 64, false>(),   make_variant<64, 64, true>(),
        make_variant<128, 128, false>(), make_variant<128, 128, true>(),
        make_variant<256, 128, false>(), make_variant<256, 128, true>(),
        make_variant<256, 256, false>(), make_variant<256, 256, true>(),
    };
    for (const Variant& v : table)
        if (v.bm == bm && v.bn == bn && v.bf16 == bf16) return &v;
    return nullptr;
}

symtile_status coresident_limit(const Variant* v, int device, int* cus, int* limit) {
    int n_cu = symtile_host::cu_count(device);
    if (n_cu <= 0) return symtile_host::fail(SYMTILE_EHIP, "cannot read the CU count");
    int per_cu = 0;
    SYMTILE_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, v->gas, kThreads, 0));
    *cus = n_cu;
    *limit = per_cu * n_cu;
    return SYMTILE_OK;
}

}  // namespace

extern "C" symtile_status symtile_device_info(int device, int tile_m, int tile_n, int* cu_count,
                                              int* max_coresident_wgs) {
    if (tile_m == 0 && tile_n == 0) tile_m = tile_n = 256;
    const Variant* v = find_variant(tile_m, tile_n, true);
    if (!v) return symtile_host::fail(SYMTILE_EUNSUPPORTED, "tile shape not built");
    int cus = 0, lim = 0;
    if (symtile_status st = coresident_limit(v, device, &cus, &lim)) return st;
    if (cu_count) *cu_count = cus;
    if (max_coresident_wgs) *max_coresident_wgs = lim;
    return SYMTILE_OK;
}

extern "C" symtile_status symtile_gemm_all_scatter(
    symtile_heap* h, const void* A, const void* B_shard, void* C_gathered_local,
    uint32_t* arrived_local, uint32_t* ready, int M, int N_local, int K, int lda, int ldb,
    int dtype, int rank, int world_size, const symtile_gas_config* cfg_in, symtile_stream s) {
    using symtile_host::fail;
    if (!h) return fail(SYMTILE_EINVAL, "heap is NULL");
    symtile_gas_config cfg{};
    if (cfg_in) cfg = *cfg_in;
    if (cfg.tile_m == 0 && cfg.tile_n == 0) cfg.tile_m = cfg.tile_n = 256;
    if (cfg.epoch == 0) cfg.epoch = 1;
    if (cfg.spin_limit == 0) cfg.spin_limit = 1u << 22;
    if (cfg.group_m <= 0) cfg.group_m = 4;
    if (cfg.variant < SYMTILE_BULK_SYNC || cfg.variant > SYMTILE_WG_SPEC)
        return fail(SYMTILE_EINVAL, "unknown variant");
    if (dtype != SYMTILE_F16 && dtype != SYMTILE_BF16)
        return fail(SYMTILE_EUNSUPPORTED, "dtype must be SYMTILE_F16 or SYMTILE_BF16");
    if (world_size != h->world) return fail(SYMTILE_EINVAL, "world_size differs from the heap's");
    if (rank < 0 || rank >= world_size) return fail(SYMTILE_EINVAL, "rank out of range");
    if (M < 0 || N_local < 0 || K < 0) return fail(SYMTILE_EINVAL, "negative size");
    if (lda == 0) lda = K;
    if (ldb == 0) ldb = N_local;
    if (lda < K || ldb < N_local) return fail(SYMTILE_EINVAL, "lda < K or ldb < N_local");
    if (K % 8 || N_local % 8 || lda % 8 || ldb % 8)
        return fail(SYMTILE_EINVAL, "K, N_local, lda and ldb must be multiples of 8");
    const Variant* v = find_variant(cfg.tile_m, cfg.tile_n, dtype == SYMTILE_BF16);
    if (!v) return fail(SYMTILE_EUNSUPPORTED, "tile shape not built");
    if ((size_t)world_size * N_local > INT32_MAX) return fail(SYMTILE_EINVAL, "N too large");
    if (M == 0 || N_local == 0) return SYMTILE_OK;   // no tiles, nothing to publish
    if ((K > 0 && (!A || !B_shard)) || !C_gathered_local || !arrived_local)
        return fail(SYMTILE_EINVAL, "NULL pointer argument");
    if (reinterpret_cast<uintptr_t>(A) % 16 || reinterpret_cast<uintptr_t>(B_shard) % 16 ||
        reinterpret_cast<uintptr_t>(C_gathered_local) % 16 ||
        reinterpret_cast<uintptr_t>(arrived_local) % 4)
        return fail(SYMTILE_EINVAL, "A, B_shard and C_gathered_local must be 16-byte aligned");

    const int tiles_m = (M + cfg.tile_m - 1) / cfg.tile_m;
    const int tiles_n = (N_local + cfg.tile_n - 1) / cfg.tile_n;
    const size_t num_tiles = (size_t)tiles_m * tiles_n;
    const size_t ldc = (size_t)world_size * N_local;
    const size_t c_bytes = ((size_t)(M - 1) * ldc + ldc) * 2;
    const size_t flag_bytes = (size_t)world_size * num_tiles * 4;
    if (!symtile_host::in_slot(h, C_gathered_local, c_bytes, rank))
        return fail(SYMTILE_EINVAL, "C_gathered_local [M, w*N_local] is not inside slot `rank`");
    if (!symtile_host::in_slot(h, arrived_local, flag_bytes, rank))
        return fail(SYMTILE_EINVAL, "arrived_local [w, tiles_m, tiles_n] is not inside slot `rank`");
    {
        const uint64_t c0 = reinterpret_cast<uint64_t>(C_gathered_local);
        const uint64_t f0 = reinterpret_cast<uint64_t>(arrived_local);
        if (f0 < c0 + c_bytes && c0 < f0 + flag_bytes)
            return fail(SYMTILE_EINVAL, "arrived_local overlaps C_gathered_local");
    }
    if (cfg.variant == SYMTILE_WG_SPEC && !ready)
        return fail(SYMTILE_EINVAL, "WG_SPEC needs a ready counter array");

    int cus = 0, limit = 0;
    if (symtile_status st = coresident_limit(v, h->device, &cus, &limit)) return st;

    GasParams p;
    p.A = static_cast<const uint16_t*>(A);
    p.B = static_cast<const uint16_t*>(B_shard);
    p.C = static_cast<uint16_t*>(C_gathered_local);
    p.arrived = arrived_local;
    p.ready = ready;
    p.bases = h->dev_bases;
    p.err = h->dev_err;
    p.M = M;
    p.N = N_local;
    p.K = K;
    p.lda = lda;
    p.ldb = ldb;
    p.ldc = (int)ldc;
    p.rank = rank;
    p.world = world_size;
    p.tiles_m = tiles_m;
    p.tiles_n = tiles_n;
    p.num_tiles = (int)num_tiles;
    p.group_m = cfg.group_m;
    p.epoch = cfg.epoch;
    p.spin_limit = cfg.spin_limit;
    p.nontemporal = cfg.nontemporal;
    p.copy_wgs = 0;

    hipStream_t stream = static_cast<hipStream_t>(s);
    int prev = -1;
    if (symtile_status st = symtile_host::set_device(h, &prev)) return st;
    struct Restore {
        int d;
        ~Restore() {
            if (d >= 0) (void)hipSetDevice(d);
        }
    } restore{prev};

    const int ntiles = (int)num_tiles;
    if (cfg.variant == SYMTILE_FUSED_SEQ || cfg.variant == SYMTILE_BULK_SYNC) {
        int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : std::min(ntiles, cus);
        g = std::min(g, ntiles);
        p.gemm_wgs = g;
        p.role = cfg.variant == SYMTILE_FUSED_SEQ ? ROLE_FUSED : ROLE_LOCAL_ONLY;
        void* args[] = {&p};
        SYMTILE_HIP(hipLaunchKernel(v->gas, dim3(g), dim3(kThreads), args, 0, stream));
        if (cfg.variant == SYMTILE_BULK_SYNC && world_size > 1) {
            int c = cfg.copy_wgs > 0 ? cfg.copy_wgs : cus;
            c = std::min(c, ntiles);
            p.copy_wgs = c;
            SYMTILE_HIP(hipLaunchKernel(v->scatter, dim3(c), dim3(kThreads), args, 0, stream));
        }
        return SYMTILE_OK;
    }

    // WG_SPEC: producers and consumers must all be resident at once.
    int c = cfg.copy_wgs > 0 ? cfg.copy_wgs : std::max(1, cus / 8);
    int g = cfg.gemm_wgs > 0 ? cfg.gemm_wgs : cus - c;
    if (g <= 0 || c <= 0) return fail(SYMTILE_EINVAL, "WG_SPEC needs gemm_wgs > 0 and copy_wgs > 0");
    if (g + c > limit)
        return fail(SYMTILE_EUNSUPPORTED,
                    "gemm_wgs + copy_wgs = " + std::to_string(g + c) +
                        " exceeds the co-resident limit " + std::to_string(limit));
    if (world_size == 1) c = std::min(c, ntiles);
    p.gemm_wgs = g;
    p.copy_wgs = c;
    p.role = ROLE_WG_SPEC;
    void* args[] = {&p};
    SYMTILE_HIP(hipLaunchKernel(v->gas, dim3(g + c), dim3(kThreads), args, 0, stream));
    return SYMTILE_OK;
}
