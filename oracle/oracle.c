/*
 * ORACLE (test infrastructure, not part of the product).
 *
 * A plain, slow, obviously correct CPU model of one rank's share of the
 * fused GEMM + All-Scatter studied in "Iris: First-Class Multi-GPU
 * Programming Experience in Triton" (arXiv 2511.12500).  Only the test
 * suite, the smoke check and the CPU-baseline leg of the benchmark may load
 * it.  It shares no code, header or table with the HIP library.
 *
 * What it models, with the passage each routine follows:
 *   - decoding of the 16-bit input formats to binary32 (inputs are rounded
 *     once on the host; the method starts from those bits);
 *   - the GEMM main loop of the paper's Section 4 GEMM listing: an fp32
 *     accumulator starts at zero and receives a[i,k]*b[k,j] for k = 0..K-1;
 *   - the gathered-output placement of Section 4.2 (fused sequential
 *     listing): rank r's tile lands at column offset r*N_local of the
 *     gathered output in every rank's heap, the rank's own heap included;
 *   - per-tile arrival counters (the counter reading of the lock protocol
 *     of the workgroup-specialised listing, Section 4.2.2);
 *   - the symmetric-heap tile copy (pointer-based put of Section 3.3.2)
 *     from every rank r to rank (r + shift) mod w.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (no fast-math,
 * so every product and sum is an individually rounded binary32 operation).
 */
#include <stdint.h>
#include <string.h>

/* ---- 16-bit formats -> binary32 ------------------------------------- */

/* bfloat16 is the upper half of an IEEE-754 binary32: sign, 8-bit exponent,
 * 7 stored mantissa bits.  Widening is exact: append 16 zero bits. */
static float bf16_bits_to_f32(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* IEEE-754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 mantissa
 * bits.  Value = (-1)^s * 2^(e-15) * (1 + m/1024) for 0 < e < 31,
 * (-1)^s * 2^-14 * (m/1024) for e = 0, inf/nan for e = 31.  Every binary16
 * value is exactly representable in binary32, so this is exact. */
static float f16_bits_to_f32(uint16_t h) {
    uint32_t sign = (uint32_t)(h >> 15) & 1u;
    uint32_t e = (uint32_t)(h >> 10) & 0x1Fu;
    uint32_t m = (uint32_t)h & 0x3FFu;
    uint32_t u;
    if (e == 0x1Fu) {                 /* inf or nan: keep payload */
        u = (sign << 31) | 0x7F800000u | (m << 13);
    } else if (e != 0) {              /* normal: rebias 15 -> 127 */
        u = (sign << 31) | ((e + 112u) << 23) | (m << 13);
    } else if (m == 0) {              /* signed zero */
        u = sign << 31;
    } else {                          /* subnormal: normalise m * 2^-24 */
        int shift = 0;
        while ((m & 0x400u) == 0) { m <<= 1; ++shift; }
        m &= 0x3FFu;
        u = (sign << 31) | ((uint32_t)(113 - shift) << 23) | (m << 13);
    }
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* dtype codes: 1 = binary16, 2 = bfloat16 */
int oracle_decode16(const uint16_t* src, float* dst, int64_t n, int dtype) {
    if (dtype != 1 && dtype != 2) return -1;
    for (int64_t i = 0; i < n; ++i)
        dst[i] = dtype == 1 ? f16_bits_to_f32(src[i]) : bf16_bits_to_f32(src[i]);
    return 0;
}

/* ---- GEMM (Section 4, GEMM main-loop listing) ------------------------ */

/* C[i,j] = sum_{k=0}^{K-1} A[i,k] * B[k,j], one binary32 accumulator per
 * output element, starting at +0 and receiving the products in increasing
 * k.  A is M x K (row stride lda), B is K x N (row stride ldb), C is M x N
 * (row stride ldc), all row-major.  The (i, k, j) loop order keeps the
 * per-element order of additions identical to the (i, j, k) definition. */
void oracle_gemm_f32(const float* A, const float* B, float* C,
                     int64_t M, int64_t N, int64_t K,
                     int64_t lda, int64_t ldb, int64_t ldc) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < M; ++i) {
        float* c = C + i * ldc;
        for (int64_t j = 0; j < N; ++j) c[j] = 0.0f;
        for (int64_t k = 0; k < K; ++k) {
            const float a = A[i * lda + k];
            const float* b = B + k * ldb;
            for (int64_t j = 0; j < N; ++j) c[j] = c[j] + a * b[j];
        }
    }
}

/* The same definition evaluated only at the n requested (row, col) pairs,
 * for spot checks at sizes where the full product is too slow. */
void oracle_gemm_entries(const float* A, const float* B, int64_t K,
                         int64_t lda, int64_t ldb,
                         const int64_t* rows, const int64_t* cols, int64_t n,
                         float* out) {
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < n; ++t) {
        float acc = 0.0f;
        for (int64_t k = 0; k < K; ++k)
            acc = acc + A[rows[t] * lda + k] * B[k * ldb + cols[t]];
        out[t] = acc;
    }
}

/* ---- placement into the gathered layout (Section 4.2, fused sequential) */

/* Rank `rank` owns columns [rank*N_local, (rank+1)*N_local) of the gathered
 * output, whose rows have w*N_local elements.  The tile is stored into
 * every rank's heap, the rank's own heap included, so for every slot s:
 *     G_s[i, rank*N_local + j] = C[i, j],  0 <= i < M, 0 <= j < N_local.
 * G is [world][M][world*N_local] float; written (same shape, bytes) gets 1
 * at every stored element.  Nothing else is touched. */
void oracle_place(const float* C, int64_t M, int64_t N_local, int world,
                  int rank, float* G, uint8_t* written) {
    const int64_t ldg = (int64_t)world * N_local;
    for (int s = 0; s < world; ++s) {
        float* g = G + (int64_t)s * M * ldg;
        uint8_t* wm = written ? written + (int64_t)s * M * ldg : 0;
        for (int64_t i = 0; i < M; ++i)
            for (int64_t j = 0; j < N_local; ++j) {
                const int64_t off = i * ldg + ((int64_t)rank * N_local + j);
                g[off] = C[i * N_local + j];
                if (wm) wm[off] = 1;
            }
    }
}

/* ---- per-tile arrival counters (Section 4.2.2, counter reading) ------ */

/* One counter per (destination slot s, source rank r, tile row m, tile
 * column n): arrived[s][r][m][n], tiles ceil(M/BM) x ceil(N_local/BN),
 * partial edge tiles counted as tiles.  One call of rank `rank` adds `inc`
 * to its counter in every slot, once per tile. */
void oracle_flags(uint32_t* arrived, int world, int rank,
                  int64_t tiles_m, int64_t tiles_n, uint32_t inc) {
    for (int s = 0; s < world; ++s)
        for (int64_t m = 0; m < tiles_m; ++m)
            for (int64_t n = 0; n < tiles_n; ++n) {
                const int64_t idx =
                    (((int64_t)s * world + rank) * tiles_m + m) * tiles_n + n;
                arrived[idx] += inc;
            }
}

/* ---- symmetric-heap tile copy (Section 3.3.2, put) -------------------- */

/* send and recv are [world][rows][cols] arrays of `esize`-byte elements
 * (row stride cols).  For every source rank r (all ranks when only_rank < 0,
 * else just only_rank) and every tile_r x tile_c tile of send[r] (partial
 * edge tiles included), the tile's bytes are copied to the same position of
 * recv[(r + shift) mod world] and that slot's counter copyflag[dst][tile] is
 * incremented by one.  copyflag is [world][tiles]. */
void oracle_tile_copy(const uint8_t* send, uint8_t* recv, uint32_t* copyflag,
                      int world, int64_t rows, int64_t cols, int esize,
                      int64_t tile_r, int64_t tile_c, int shift, int only_rank, int get) {
    const int64_t tiles_r = (rows + tile_r - 1) / tile_r;
    const int64_t tiles_c = (cols + tile_c - 1) / tile_c;
    const int64_t slot_bytes = rows * cols * esize;
    for (int r = 0; r < world; ++r) {
        if (only_rank >= 0 && r != only_rank) continue;
        /* put: rank r writes its send into rank r+shift's recv;
           get: rank r reads rank r-shift's send into its own recv */
        const int src = get ? ((r - shift) % world + world) % world : r;
        const int dst = get ? r : ((r + shift) % world + world) % world;
        for (int64_t tr = 0; tr < tiles_r; ++tr)
            for (int64_t tc = 0; tc < tiles_c; ++tc) {
                for (int64_t i = tr * tile_r; i < rows && i < (tr + 1) * tile_r; ++i)
                    for (int64_t j = tc * tile_c; j < cols && j < (tc + 1) * tile_c; ++j) {
                        const int64_t e = (i * cols + j) * esize;
                        memcpy(recv + dst * slot_bytes + e, send + src * slot_bytes + e,
                               (size_t)esize);
                    }
                copyflag[(int64_t)dst * tiles_r * tiles_c + tr * tiles_c + tc] += 1u;
            }
    }
}
