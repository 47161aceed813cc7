// Pool scan: s[b][i] = q_b . k_i for every stored position i < n_valid
// (Algorithm 1 retrieve step; with unit operands this is cos(h_t, h_i)).
// bf16 operands, fp32 accumulation.  The key pool is read exactly once per
// call.  The scan keeps, per (query, 32-row block), only the block's best
// (score, position) key; the top-k passes pick the k best blocks per query
// and the rescore kernels below recompute those blocks' 32 scores with the
// scan's own instruction sequence (bit-identical values).  Writing every
// score (B x N x 4 bytes) interleaves a large store stream with the key reads
// and costs far more than its bytes; re-reading k blocks per query does not.
//
// The pool is stored as 4 KiB tiles (32 rows x 64 columns) in MFMA operand
// order, window-major (see store.hip): every 16-byte-per-lane load reads
// 1 KiB contiguous, and while the waves walk their row blocks window by
// window the chip reads one contiguous region at a time, the access pattern
// of a plain copy.
//
// Kernels, chosen by the query batch:
//  * scan_gemv (B <= 4): a matrix-vector product on the vector ALU
//    (v_dot2 bf16 -> fp32).  Lane l accumulates row l % 32 of the tile over
//    half of each window's columns; one xor-32 exchange completes the row.
//    Queries sit in LDS, read as broadcasts.  It runs on small pools only (B *
//    N at most 2^19 scores), where it also writes every score: the final
//    selection reads the chosen blocks' scores from there, and no rescore
//    runs.  On larger pools those writes, interleaved with the key stream,
//    would cost the scan more than a rescore (1M positions: +25 us at B = 1,
//    +73 us at B = 4), and the MFMA scan, its 32-query tile mostly empty,
//    reads the pool faster than the GEMV without them (1.208 / 1.207 ms at
//    B = 1 / 4 against 1.232 / 1.250), so it takes those batches.
//  * scan_mfma (B <= 64): the batch makes the scan a dense contraction;
//    v_mfma_f32_32x32x16_bf16 multiplies a 32-key tile by a 32-query tile
//    fragment per instruction, the fragments pre-swizzled by query prep.
//  * scan_mfma_wide (64 < B <= 512): the same instruction, keys shared by all
//    query tiles through LDS (the contraction turns MFMA-bound near B ~ 300).
//  * scan_mfma_persist (bf16 keys, B <= 32, pools of two or more whole
//    rounds of its groups): scan_mfma as a persistent grid whose waves
//    stream from one group of row blocks into the next.
//  * scan_tail (remainder of the B <= 64 scan): the few row blocks past its
//    last whole generation of waves, one workgroup each, through a deep LDS
//    ring.
//
// The first two run a software pipeline: a ring of PF + 1 register stages,
// window w + PF requested before window w is consumed.  Loads are
// unconditional (window index clamped; the repeats at the end hit in cache)
// so the compiler counts outstanding loads exactly.  The wide scan pipelines
// through LDS instead (below).
//
// Tile (row block rb, window w) starts at element rb * rs + w * ws, so the
// kernels serve both tile orders (row-block-major and window-major).
//
// A key's accumulation order never depends on where the key sits, so
// identical keys score identically.  Positions whose prompt id equals the
// query's exclusion id get the "no position" bit pattern.
#include <hip/hip_ext.h>

#include <numeric>
#include <utility>

#include "common.hpp"
#include "internal.hpp"

// Row blocks per wave and prefetch depth of the scans for B <= 64.
#ifndef OIL_BF16_MT
#define OIL_BF16_MT 4
#endif
#ifndef OIL_BF16_PF
#define OIL_BF16_PF 1
#endif
#ifndef OIL_FP8_MT
#define OIL_FP8_MT 2
#endif
// Row blocks per wave for two query tiles (33 <= B <= 64).
#ifndef OIL_BF16_MT2
#define OIL_BF16_MT2 OIL_BF16_MT
#endif
#ifndef OIL_FP8_MT2
#define OIL_FP8_MT2 4
#endif
#ifndef OIL_FP8_PF
#define OIL_FP8_PF 1
#endif
// Prefetch depth (windows in flight per wave) of the MFMA rescore.  At 1M x
// 4096, B = k = 32 (1024 waves, one per SIMD): depth 0 73 us, 1 45, 2 46, 3 47.5.
#ifndef OIL_RESCORE_PF
#define OIL_RESCORE_PF 1
#endif
// Windows in flight per wave of the remainder launch of the B <= 64 scan,
// for one and two query tiles.
#ifndef OIL_TAIL_PF1
#define OIL_TAIL_PF1 7
#endif
#ifndef OIL_TAIL_PF2
#define OIL_TAIL_PF2 3
#endif
// Remainders of up to one row block per compute unit past the B <= 64
// scan's whole generations of waves go to scan_tail_kernel (0: never).
#ifndef OIL_TAIL_LDS
#define OIL_TAIL_LDS 1
#endif
// The bf16 B <= 32 scan runs as a persistent kernel over whole rounds of its
// groups (0: one workgroup per group; PERSIST_FP8: fp8 keys too).
#ifndef OIL_SCAN_PERSIST
#define OIL_SCAN_PERSIST 1
#endif
#ifndef OIL_SCAN_PERSIST_PART
#define OIL_SCAN_PERSIST_PART 1
#endif
#ifndef OIL_SCAN_PERSIST_FP8
#define OIL_SCAN_PERSIST_FP8 0
#endif
// Cache policy of the wide scan's key copies: 2 = nt (streaming, as the
// narrow scans' nontemporal key loads).
#ifndef OIL_WIDE_KEY_CPOL
#define OIL_WIDE_KEY_CPOL 2
#endif

namespace oil {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// acc + sum of the 8 products a[e] * b[e] (four v_dot2 bf16 -> fp32 steps, in order).
__device__ __forceinline__ float dot8_bf16(const bf16x8 a, const bf16x8 b, float acc)
{
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1),
                                          __builtin_shufflevector(b, b, 0, 1), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3),
                                          __builtin_shufflevector(b, b, 2, 3), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5),
                                          __builtin_shufflevector(b, b, 4, 5), acc, false);
    acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7),
                                          __builtin_shufflevector(b, b, 6, 7), acc, false);
    return acc;
}

__device__ __forceinline__ float masked_score(float s, int64_t row, int32_t ex,
                                              const int32_t* __restrict__ prompt)
{
    if (ex >= 0 && prompt[row] == ex)
        return __uint_as_float(kNoScoreBits);
    return s;
}

// Per-row data (inverse key scales, prompt ids) of the 16 rows a lane holds
// in a 32-row MFMA tile starting at row0: element 4 i + j is row
// row0 + 8 i + 4 h + j.  The 16 loads are issued together; indices past the
// last stored row are clamped to it (those rows are never scored).
template <typename T>
__device__ __forceinline__ void tile_rows_load(T (&out)[16], const T* __restrict__ src, int64_t row0, int h,
                                               int64_t n_valid)
{
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int64_t row = row0 + i * 8 + h * 4 + j;
            out[4 * i + j] = src[row < n_valid ? row : n_valid - 1];
        }
}

// ----------------------------------------------------------------- GEMV (B <= 4)
template <int NB, int PF>
__global__ __launch_bounds__(256) void scan_gemv_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const uint16_t* __restrict__ q, const int32_t* __restrict__ prompt,
    const int32_t* __restrict__ exclude, uint64_t* __restrict__ G, int64_t g_ld, float* __restrict__ FS,
    int64_t fs_ld)
{
    constexpr int NS = PF + 1;
    extern __shared__ __align__(16) uint16_t q_lds[];  // NB x ld, row-major
    for (int64_t j = threadIdx.x * 8; j < (int64_t)NB * ld; j += 256 * 8)
        *(bf16x8*)(q_lds + j) = *(const bf16x8*)(q + j);
    __syncthreads();

    const int lane = threadIdx.x & 63;
    const int h = lane >> 5, r = lane & 31;
    const int64_t rb = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (rb * kRowBlock >= n_valid)
        return;
    const int nwin = ld / kWindow;
    const bf16x8* tile = (const bf16x8*)(keys + rb * rs) + lane;
    const int64_t ws8 = ws / 8;

    float acc[NB];
#pragma unroll
    for (int b = 0; b < NB; b++)
        acc[b] = 0.f;
    bf16x8 a[NS][4];
#pragma unroll
    for (int p = 0; p < PF; p++) {
        const int w = p < nwin ? p : nwin - 1;
#pragma unroll
        for (int s = 0; s < 4; s++)
            a[p][s] = __builtin_nontemporal_load(tile + w * ws8 + s * 64);
    }
    const int nloop = (nwin + NS - 1) / NS * NS;
    for (int w0 = 0; w0 < nloop; w0 += NS) {
#pragma unroll
        for (int u = 0; u < NS; u++) {
            const int wl = w0 + u + PF < nwin ? w0 + u + PF : nwin - 1;
#pragma unroll
            for (int s = 0; s < 4; s++)
                a[(u + PF) % NS][s] = __builtin_nontemporal_load(tile + wl * ws8 + s * 64);
            if (w0 + u < nwin) {
                const int col = (w0 + u) * kWindow + 32 * h;
#pragma unroll
                for (int s = 0; s < 4; s++)
#pragma unroll
                    for (int b = 0; b < NB; b++)
                        acc[b] = dot8_bf16(a[u][s], *(const bf16x8*)(q_lds + b * ld + col + 8 * s),
                                           acc[b]);
            }
        }
    }
    // Lanes r and r + 32 now both hold row r's full score: lane r stores it,
    // and each query keeps the best (score, position) key of this row block.
    const int64_t row = rb * kRowBlock + r;
#pragma unroll
    for (int b = 0; b < NB; b++) {
        const float full = acc[b] + __shfl_xor(acc[b], 32, kWave);
        const int32_t ex = exclude ? exclude[b] : -1;
        const bool have = row < n_valid;
        const float v = have ? masked_score(full, row, ex, prompt) : 0.f;
        if (FS && have && h == 0)
            FS[b * fs_ld + row] = v;
        uint64_t best = have ? rank_key(v, (uint32_t)row) : 0ull;
#pragma unroll
        for (int o = 16; o >= 1; o >>= 1) {
            const uint64_t other = __shfl_xor(best, o, kWave);
            best = other > best ? other : best;
        }
        if (lane == 0)
            G[b * g_ld + rb] = best;
    }
}

// ----------------------------------------------------------------- MFMA (4 < B <= 64)
// One 16-byte operand register per lane and sub-step: eight bf16 (one
// 32x32x16 bf16 MFMA), or sixteen OCP E4M3 values of a 128-column fp8 window
// (two sub-steps per fp8 MFMA, below).
__device__ __forceinline__ floatx16 mfma_step(const bf16x8& a, const bf16x8& b, floatx16 acc)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}

// fp8 keys: two 16-byte sub-steps (32 fp8 values per lane, for keys and
// queries alike) feed one v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales
// (E8M0 127 = 2^0).  Keys and query fragments share one tile layout, so
// operand slot j of a lane holds the same column for both: the instruction's
// own k order pairs every key column with its query column.
__device__ __forceinline__ floatx16 mfma_pair_fp8(const bf16x8& a0, const bf16x8& a1, const bf16x8& b0,
                                                  const bf16x8& b1, floatx16 acc)
{
    typedef int int4v __attribute__((ext_vector_type(4)));
    typedef int int8v __attribute__((ext_vector_type(8)));
    const int4v x0 = __builtin_bit_cast(int4v, a0), x1 = __builtin_bit_cast(int4v, a1);
    const int4v y0 = __builtin_bit_cast(int4v, b0), y1 = __builtin_bit_cast(int4v, b1);
    const int8v a = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
    const int8v b = {y0[0], y0[1], y0[2], y0[3], y1[0], y1[1], y1[2], y1[3]};
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, acc, 0, 0, 0, 127, 0, 127);
}

template <int MT, int NT>
__device__ __forceinline__ void load_window(bf16x8 (&a)[MT][4], bf16x8 (&b)[NT][4],
                                            const bf16x8* const (&tile)[MT], int64_t ws8,
                                            const bf16x8* __restrict__ qf, int w)
{
#pragma unroll
    for (int mt = 0; mt < MT; mt++)
#pragma unroll
        for (int s = 0; s < 4; s++)
            a[mt][s] = __builtin_nontemporal_load(tile[mt] + w * ws8 + s * 64);
#pragma unroll
    for (int nt = 0; nt < NT; nt++)
#pragma unroll
        for (int s = 0; s < 4; s++)
            b[nt][s] = qf[(((int64_t)w * NT + nt) * 4 + s) * 64];
}

template <int MT, int NT, int PF, int FMT>
__global__ __launch_bounds__(256) void scan_mfma_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const bf16x8* __restrict__ qfrag, int32_t B, const int32_t* __restrict__ prompt,
    const int32_t* __restrict__ exclude, uint64_t* __restrict__ G, int64_t g_ld,
    const float* __restrict__ kscale, const float* __restrict__ qscale, int64_t rb_base)
{
    constexpr int NS = PF + 1;
    const int lane = threadIdx.x & 63;
    const int h = lane >> 5, r = lane & 31;
    const int wave = threadIdx.x >> 6;
    const int64_t rbb = rb_base + (int64_t)blockIdx.x * 4 * MT;  // the block's first row block
    const int64_t rb0 = rbb + wave * MT;
    const bool live = rb0 * kRowBlock < n_valid;  // waves past the pool only join the block store
    const int64_t n_rb = (n_valid + kRowBlock - 1) / kRowBlock;
    const int nwin = ld / (FMT == kKeyBf16 ? kWindow : kWindowFp8);
    const int64_t ws8 = ws / 8;

    const bf16x8* tile[MT];
#pragma unroll
    for (int mt = 0; mt < MT; mt++) {
        const int64_t rb = rb0 + mt < n_rb ? rb0 + mt : n_rb - 1;  // clamp: stays inside the pool
        tile[mt] = (const bf16x8*)(keys + rb * rs) + lane;
    }
    const bf16x8* qf = qfrag + lane;

    floatx16 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; mt++)
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
            acc[mt][nt] = floatx16{};

    bf16x8 a[NS][MT][4], b[NS][NT][4];
#pragma unroll
    for (int p = 0; p < PF; p++)
        load_window<MT, NT>(a[p], b[p], tile, ws8, qf, p < nwin ? p : nwin - 1);
    const int nloop = live ? (nwin + NS - 1) / NS * NS : 0;
    for (int w0 = 0; w0 < nloop; w0 += NS) {
#pragma unroll
        for (int u = 0; u < NS; u++) {
            const int wl = w0 + u + PF < nwin ? w0 + u + PF : nwin - 1;
            load_window<MT, NT>(a[(u + PF) % NS], b[(u + PF) % NS], tile, ws8, qf, wl);
            if (w0 + u < nwin) {
                if constexpr (FMT == kKeyFp8) {
#pragma unroll
                    for (int s = 0; s < 4; s += 2)
#pragma unroll
                        for (int mt = 0; mt < MT; mt++)
#pragma unroll
                            for (int nt = 0; nt < NT; nt++)
                                acc[mt][nt] = mfma_pair_fp8(a[u][mt][s], a[u][mt][s + 1], b[u][nt][s],
                                                            b[u][nt][s + 1], acc[mt][nt]);
                } else {
#pragma unroll
                    for (int s = 0; s < 4; s++)
#pragma unroll
                        for (int mt = 0; mt < MT; mt++)
#pragma unroll
                            for (int nt = 0; nt < NT; nt++)
                                acc[mt][nt] = mfma_step(a[u][mt][s], b[u][nt][s], acc[mt][nt]);
                }
            }
        }
    }

    // Accumulator layout of a 32x32 MFMA tile: lane l, element 4 i + j holds
    // row 8 i + 4 (l / 32) + j (a key) and column l % 32 (a query).  Each
    // (query, row block) keeps its best (score, position) key.  The keys of
    // the block's 4 MT row blocks are gathered in LDS and stored by the whole
    // block, row by row (consecutive threads, consecutive row blocks of one
    // query: 4 MT keys per query row) instead of one scattered 8-byte store
    // per query (~30 us more at 1M x 4096, B = 32) or one segment per wave
    // (6 us more).  The stores are non-temporal (streamed past the caches the
    // key stream uses): at 1M x 4096, B = 32 the persistent scan takes
    // 1,215 us against 1,224 with plain stores.
    __shared__ uint64_t gk[4][NT * 32][MT + 1];  // per wave; +1: rows land in different banks
    int32_t ex[NT];
    float qs[NT];
#pragma unroll
    for (int nt = 0; nt < NT; nt++) {
        const int qb = nt * 32 + r;
        const bool qlive = qb < B;
        ex[nt] = (exclude && qlive) ? exclude[qb] : -1;
        qs[nt] = (FMT == kKeyBf16 || !qlive) ? 1.f : qscale[qb];
    }
#pragma unroll
    for (int mt = 0; mt < MT; mt++) {
        const int64_t rb = rb0 + mt;
        float ks[16];
        int32_t pr[16];
        if constexpr (FMT == kKeyFp8)
            tile_rows_load(ks, kscale, rb * kRowBlock, h, n_valid);
        if (exclude)
            tile_rows_load(pr, prompt, rb * kRowBlock, h, n_valid);
#pragma unroll
        for (int nt = 0; nt < NT; nt++) {
            uint64_t best = 0;
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int64_t row = rb * kRowBlock + (e / 4) * 8 + h * 4 + e % 4;
                if (row < n_valid) {
                    float v = acc[mt][nt][e];
                    if constexpr (FMT == kKeyFp8)
                        v = v * (ks[e] * qs[nt]);  // powers of two: exact
                    if (ex[nt] >= 0 && pr[e] == ex[nt])
                        v = __uint_as_float(kNoScoreBits);
                    const uint64_t key = rank_key(v, (uint32_t)row);
                    best = key > best ? key : best;
                }
            }
            const uint64_t other = __shfl_xor(best, 32, kWave);
            best = other > best ? other : best;
            if (h == 0)
                gk[wave][nt * 32 + r][mt] = best;
        }
    }
    __syncthreads();
    const int nq = B < NT * 32 ? B : NT * 32;
    constexpr int KPB = 4 * MT;  // the block's keys per query
#pragma unroll
    for (int c0 = 0; c0 < NT * 32 * KPB; c0 += 256) {
        const int c = c0 + (int)threadIdx.x;
        const int q = c / KPB, j = c % KPB;
        if (q < nq && rbb + j < n_rb)
            __builtin_nontemporal_store(gk[j / MT][q][j % MT], &G[q * g_ld + rbb + j]);
    }
}

// Persistent form of scan_mfma_kernel for one query tile: a grid of as many
// workgroups as the chip holds at once walks groups g, g + grid, ... of 4 MT
// row blocks (a whole number of rounds).  Each wave requests the next group's
// first window during the current group's last one, and the epilogue's
// barriers wait for LDS only, so the key stream does not drain between groups
// as it does when a workgroup ends and the next one starts (1M x 4096, B = 32:
// 1.255 -> 1.239 ms).  Per row block the MFMA sequence is the scan's.
template <int MT, int NT, int FMT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NT == 1 ? 2 : 1))) void scan_mfma_persist_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const bf16x8* __restrict__ qfrag, int32_t B, const int32_t* __restrict__ prompt,
    const int32_t* __restrict__ exclude, uint64_t* __restrict__ G, int64_t g_ld,
    const float* __restrict__ kscale, const float* __restrict__ qscale, int64_t n_groups)
{
    constexpr int NS = 2;
    const int lane = threadIdx.x & 63;
    const int h = lane >> 5, r = lane & 31;
    const int wave = threadIdx.x >> 6;
    const int64_t n_rb = (n_valid + kRowBlock - 1) / kRowBlock;
    const int nwin = ld / (FMT == kKeyBf16 ? kWindow : kWindowFp8);
    const int64_t ws8 = ws / 8;
    const int64_t stride = gridDim.x;
    int64_t g = blockIdx.x;
    if (g >= n_groups)
        return;
    // tiles as offsets from the pool's base (16-byte units), so every load
    // keeps the global address space (pointers carried across the group
    // switch would become flat accesses, which also count as LDS accesses)
    const bf16x8* kv = (const bf16x8*)keys;
    auto tiles_of = [&](int64_t gg, int64_t (&t)[MT]) {
        const int64_t rb0 = gg * 4 * MT + wave * MT;
#pragma unroll
        for (int mt = 0; mt < MT; mt++) {
            const int64_t rb = rb0 + mt < n_rb ? rb0 + mt : n_rb - 1;  // clamp: stays inside the pool
            t[mt] = rb * rs / 8 + lane;
        }
    };
    auto load = [&](bf16x8 (&av)[MT][4], bf16x8 (&bv)[NT][4], const int64_t (&t)[MT], int w) {
#pragma unroll
        for (int mt = 0; mt < MT; mt++)
#pragma unroll
            for (int s = 0; s < 4; s++)
                av[mt][s] = __builtin_nontemporal_load(kv + t[mt] + w * ws8 + s * 64);
#pragma unroll
        for (int nt = 0; nt < NT; nt++)
#pragma unroll
            for (int s = 0; s < 4; s++)
                bv[nt][s] = qfrag[(((int64_t)w * NT + nt) * 4 + s) * 64 + lane];
    };
    int64_t cur[MT];
    tiles_of(g, cur);
    bf16x8 a[NS][MT][4], b[NS][NT][4];
    load(a[0], b[0], cur, 0);
    __shared__ uint64_t gk[4][NT * 32][MT + 1];
    for (; g < n_groups; g += stride) {
        floatx16 acc[MT][NT];
#pragma unroll
        for (int mt = 0; mt < MT; mt++)
#pragma unroll
            for (int nt = 0; nt < NT; nt++)
                acc[mt][nt] = floatx16{};
        for (int w0 = 0; w0 < nwin; w0 += NS) {
#pragma unroll
            for (int u = 0; u < NS; u++) {
                const int wl = w0 + u + 1;
                if (wl == nwin)  // the next group's tiles (this group's loads are all issued)
                    tiles_of(g + stride < n_groups ? g + stride : g, cur);
                load(a[(u + 1) % NS], b[(u + 1) % NS], cur, wl < nwin ? wl : 0);
                if constexpr (FMT == kKeyFp8) {
#pragma unroll
                    for (int s = 0; s < 4; s += 2)
#pragma unroll
                        for (int mt = 0; mt < MT; mt++)
#pragma unroll
                            for (int nt = 0; nt < NT; nt++)
                                acc[mt][nt] = mfma_pair_fp8(a[u][mt][s], a[u][mt][s + 1], b[u][nt][s],
                                                            b[u][nt][s + 1], acc[mt][nt]);
                } else {
#pragma unroll
                    for (int s = 0; s < 4; s++)
#pragma unroll
                        for (int mt = 0; mt < MT; mt++)
#pragma unroll
                            for (int nt = 0; nt < NT; nt++)
                                acc[mt][nt] = mfma_step(a[u][mt][s], b[u][nt][s], acc[mt][nt]);
                }
            }
        }
        // block keys of group g, as in scan_mfma_kernel
        const int64_t rbb = g * 4 * MT;
        const int64_t rb0 = rbb + wave * MT;
        int32_t ex[NT];
        float qs[NT];
#pragma unroll
        for (int nt = 0; nt < NT; nt++) {
            const int qb = nt * 32 + r;
            const bool qlive = qb < B;
            ex[nt] = (exclude && qlive) ? exclude[qb] : -1;
            qs[nt] = (FMT == kKeyBf16 || !qlive) ? 1.f : qscale[qb];
        }
#pragma unroll
        for (int mt = 0; mt < MT; mt++) {
            const int64_t rb = rb0 + mt;
            float ks[16];
            int32_t pr[16];
            if constexpr (FMT == kKeyFp8)
                tile_rows_load(ks, kscale, rb * kRowBlock, h, n_valid);
            if (exclude)
                tile_rows_load(pr, prompt, rb * kRowBlock, h, n_valid);
#pragma unroll
            for (int nt = 0; nt < NT; nt++) {
                uint64_t best = 0;
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const int64_t row = rb * kRowBlock + (e / 4) * 8 + h * 4 + e % 4;
                    if (row < n_valid) {
                        float v = acc[mt][nt][e];
                        if constexpr (FMT == kKeyFp8)
                            v = v * (ks[e] * qs[nt]);
                        if (ex[nt] >= 0 && pr[e] == ex[nt])
                            v = __uint_as_float(kNoScoreBits);
                        const uint64_t key = rank_key(v, (uint32_t)row);
                        best = key > best ? key : best;
                    }
                }
                const uint64_t other = __shfl_xor(best, 32, kWave);
                best = other > best ? other : best;
                if (h == 0)
                    gk[wave][nt * 32 + r][mt] = best;
            }
        }
        // LDS only: the next group's first window stays in flight
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_s_barrier();
        const int nq = B < NT * 32 ? B : NT * 32;
        constexpr int KPB = 4 * MT;
#pragma unroll
        for (int c0 = 0; c0 < NT * 32 * KPB; c0 += 256) {
            const int c = c0 + (int)threadIdx.x;
            const int q = c / KPB, j = c % KPB;
            if (q < nq && rbb + j < n_rb)
                __builtin_nontemporal_store(gk[j / MT][q][j % MT], &G[q * g_ld + rbb + j]);
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);
        __builtin_amdgcn_s_barrier();  // gk is free for the next group
    }
}

// ----------------------------------------------------------------- MFMA, wide batches (64 < B <= 512)
// Past ~300 queries the contraction is MFMA-bound, so keys must be fetched
// once and reused by every query tile.  A block owns MT row blocks; its WAVES
// waves split the query tiles (NTW tiles each) and, in groups of RS, the row
// blocks (MT / RS each: more waves share a key window without more
// accumulation registers per wave).  Each key window of the block
// (MT tiles of 4 KiB) lands in LDS once, in an R-window ring, shared by every
// wave, with 16-byte buffer loads straight to LDS (each wave copies 4 MT /
// WAVES of the block's 1 KiB chunks; loading the keys through registers and
// storing them to LDS measured slower).  Every wave reads its A operands from LDS (lane l's 16 bytes sit at 16 l:
// conflict-free) and its own query fragments from L2 into registers, NB - 1
// windows ahead.  Per (row block, query tile) the MFMA sequence is the same
// as in scan_mfma_kernel (windows in order, sub-steps in order), so scores
// are bit-identical to the narrow scan's and the rescore's.
//
// Schedule of window w (NG MFMA groups: four bf16 sub-steps, or two fp8
// pairs).  The A operands of group g + 1 are read from LDS while group g's
// MFMAs run; the fragments of window w + NB - 1 are requested between the
// MFMAs of the first NG - 1 groups (one load every few MFMAs: a burst of
// loads ahead of the MFMAs would hold up their issue).  Before the last group
// each wave makes sure its part of window w + 1 is in LDS (it waits for the
// copies it issued R - 2 windows earlier), and the waves meet at one
// barrier: window w + 1 is then in LDS, and every wave has finished reading
// window w - 1, whose slot receives the copies of window w + R - 1, issued
// between the last group's MFMAs.  The first A operands of window w + 1 are
// read right after the barrier, so the last group's MFMAs hide the LDS
// latency.  Loads past the last window repeat the last window (clamped index:
// uniform wait counts; the repeats land in a free slot or hit in cache).
//
// A workgroup barrier without the memory fence __syncthreads() carries: that
// fence would wait for every outstanding copy to LDS, the ones meant to stay
// in flight included.  The scheduling barriers keep LDS accesses on their
// side of it.
__device__ __forceinline__ void block_barrier()
{
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Waves per SIMD the wide scan's registers allow: two with at most 4 row
// blocks and 2 query tiles (bf16) or 1 tile (fp8, whose pairs hold twice the
// A operands).
#ifndef OIL_WIDE_WPE
#define OIL_WIDE_WPE(MT, NTW, FMT) ((MT) <= 4 && (NTW) <= ((FMT) == kKeyBf16 ? 2 : 1) ? 2 : 1)
#endif

template <int N>
__device__ __forceinline__ void wait_vmcnt_at_most()
{
    // s_waitcnt: vmcnt[3:0] | expcnt[6:4] | lgkmcnt[11:8] | vmcnt[5:4] << 14;
    // expcnt and lgkmcnt at their maxima (no wait on them).
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// f(std::integral_constant<int, 0>{}), ..., f(std::integral_constant<int, N - 1>{}), in order.
template <int... I, class F>
__device__ __forceinline__ void unrolled_impl(std::integer_sequence<int, I...>, F&& f)
{
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void unrolled(F&& f)
{
    unrolled_impl(std::make_integer_sequence<int, N>{}, f);
}

template <int MT, int NTW, int R, int NB, int WAVES, int WPE, int FMT, int RS, int SKIP>
__global__ __launch_bounds__(64 * WAVES) __attribute__((amdgpu_waves_per_eu(WPE))) void
scan_mfma_wide_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const bf16x8* __restrict__ qfrag, int32_t B, const int32_t* __restrict__ prompt,
    const int32_t* __restrict__ exclude, uint64_t* __restrict__ G, int64_t g_ld,
    const float* __restrict__ kscale, const float* __restrict__ qscale)
{
    constexpr int NG = FMT == kKeyBf16 ? 4 : 2;  // MFMA groups per window
    constexpr int CG = 4 / NG;                   // 1 KiB operand chunks per group
    constexpr int MTW = MT / RS;                 // row blocks per wave (RS waves share a tile group)
    static_assert(MTW * RS == MT && WAVES % RS == 0, "row split");
    constexpr int NM = MTW * NTW;                // MFMAs per group
    constexpr int NQ = NTW * 4;                  // fragment loads per window
    constexpr int CPW = 4 * MT / WAVES;          // 1 KiB key copies per wave and window
    static_assert(CPW * WAVES == 4 * MT && (NB == 2 || NB == 3), "copy split / fragment sets");
    // loads a wave may have in flight once the copies of window w + 1 are in
    // (see the schedule above)
    constexpr int kInFlight = (R - 3) * (NQ + CPW) + NQ;
    static_assert(R >= 4 && R <= 6 && kInFlight <= 63, "ring depth / vmcnt range");
    // stages per trip: ring slot and fragment set return to their start
    constexpr int U = R * NB / std::gcd(R, NB);
    // R windows of the block's MT key tiles, as separate LDS objects so that
    // the slot each access uses is known at compile time (unused ones vanish)
    __shared__ bf16x8 ring0[MT][4][64], ring1[MT][4][64], ring2[MT][4][64], ring3[MT][4][64],
        ring4[MT][4][64], ring5[MT][4][64];
    auto slot = [&](auto s_t) -> bf16x8 (&)[MT][4][64] {
        constexpr int s = decltype(s_t)::value;
        if constexpr (s == 0) return ring0;
        else if constexpr (s == 1) return ring1;
        else if constexpr (s == 2) return ring2;
        else if constexpr (s == 3) return ring3;
        else if constexpr (s == 4) return ring4;
        else return ring5;
    };
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
    const int h = lane >> 5, r = lane & 31;
    const int rp = wave % RS, tg = wave / RS;  // the wave's row part and tile group
    const int64_t rb0 = (int64_t)blockIdx.x * MT;
    const int64_t n_rb = (n_valid + kRowBlock - 1) / kRowBlock;
    const int nwin = ld / (FMT == kKeyBf16 ? kWindow : kWindowFp8);
    const int n_qt = (B + 31) / 32;
    // Addresses are a wave-uniform base plus the lane's 16-byte slot, so the
    // loads take a scalar base and one shared 32-bit lane offset.
    const uint32_t loff = (uint32_t)lane * 16;

    // this wave's share of the block's key copies: jobs j = wave + WAVES c
    // (c < CPW), job j being 1 KiB chunk j % 4 of tile j / 4
    const char* src[CPW];
    uint32_t dst[CPW];  // byte offset of the job's chunk inside a ring slot
#pragma unroll
    for (int c = 0; c < CPW; c++) {
        const int j = wave + WAVES * c;
        const int64_t rb = rb0 + j / 4 < n_rb ? rb0 + j / 4 : n_rb - 1;  // clamp: stays inside the pool
        src[c] = (const char*)(keys + rb * rs) + (j % 4) * 1024;
        dst[c] = (uint32_t)j * 1024;
    }
    const int64_t wbytes = ws * 2;
    auto clampw = [&](int w) { return w < nwin ? w : nwin - 1; };
    // Buffer (not global) loads to LDS: the compiler's wait-count tracking
    // treats a pending global-to-LDS load as a flat access and then waits for
    // every outstanding load at each register use; buffer loads keep precise
    // counts.  The descriptor's base is the tile's 1 KiB chunk (wave-uniform).
    auto copy_one = [&](bf16x8 (&buf)[MT][4][64], int c, int w) {
        const __amdgpu_buffer_rsrc_t rsrc =
            __builtin_amdgcn_make_buffer_rsrc((void*)(src[c] + w * wbytes), (short)0, 1024, 0x00020000);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            rsrc, (void __attribute__((address_space(3)))*)((char*)&buf[0][0][0] + dst[c]), 16, loff, 0, 0, OIL_WIDE_KEY_CPOL);
    };
    int qt[NTW];
#pragma unroll
    for (int nt = 0; nt < NTW; nt++) {
        const int t = tg * NTW + nt;
        qt[nt] = t < n_qt ? t : n_qt - 1;  // clamp: idle tiles recompute a live one, never stored
    }
    // fragment load l: sub-step l / NTW of tile l % NTW (the first group's
    // fragments are requested first)
    auto load_q1 = [&](bf16x8 (&b)[NTW][4], int l, int w) {
        const int nt = l % NTW, s = l / NTW;
        const char* base = (const char*)(qfrag + (((int64_t)w * n_qt + qt[nt]) * 4 + s) * 64);
        b[nt][s] = *(const bf16x8*)(base + loff);
    };

    floatx16 acc[MTW][NTW];
#pragma unroll
    for (int mt = 0; mt < MTW; mt++)
#pragma unroll
        for (int nt = 0; nt < NTW; nt++)
            acc[mt][nt] = floatx16{};

    // A operands: two register sets, one group each
    bf16x8 a[2][CG][MTW];
    auto read_group = [&](bf16x8 (&dst)[CG][MTW], const bf16x8 (&buf)[MT][4][64], int g) {
#pragma unroll
        for (int c = 0; c < CG; c++)
#pragma unroll
            for (int mt = 0; mt < MTW; mt++)
                dst[c][mt] = buf[rp * MTW + mt][g * CG + c][lane];
    };
    // MFMA i of group g: row block i / NTW, query tile i % NTW
    // SKIP (batches that leave the class's last tiles empty): those tiles
    // skip their MFMAs (a scalar branch each, which costs full batches up to
    // 5%, hence a separate instantiation)
    bool tlive[NTW];
#pragma unroll
    for (int nt = 0; nt < NTW; nt++)
        tlive[nt] = tg * NTW + nt < n_qt;  // wave-uniform
    auto mfma_one = [&](const bf16x8 (&av)[CG][MTW], const bf16x8 (&b)[NTW][4], int g, int i) {
        const int mt = i / NTW, nt = i % NTW;
        if (!SKIP || tlive[nt]) {
            if constexpr (FMT == kKeyFp8)
                acc[mt][nt] = mfma_pair_fp8(av[0][mt], av[1][mt], b[nt][2 * g], b[nt][2 * g + 1], acc[mt][nt]);
            else
                acc[mt][nt] = mfma_step(av[0][mt], b[nt][g], acc[mt][nt]);
        }
    };

    bf16x8 b0[NTW][4], b1[NTW][4], b2[NTW][4];
    auto fset = [&](auto s_t) -> bf16x8 (&)[NTW][4] {
        constexpr int s = decltype(s_t)::value;
        if constexpr (s == 0) return b0;
        else if constexpr (s == 1) return b1;
        else return b2;
    };
    // Window w = w0 + I (I a compile-time stage index) sits in slot I % R;
    // window w + 1 in slot (I + 1) % R; the copies of window w + R - 1 go to
    // slot (I + R - 1) % R, which held window w - 1.  Window w's fragments
    // are in set I % NB; the fragments of window w + NB - 1 go to set
    // (I + NB - 1) % NB, which held window w - 1's.  On entry a[0] holds
    // group 0 of window w (read issued).
    auto stage = [&](auto i_t, int w) __attribute__((always_inline)) {
        constexpr int I = decltype(i_t)::value;
        const bf16x8(&cur)[MT][4][64] = slot(std::integral_constant<int, I % R>{});
        const bf16x8(&nx1)[MT][4][64] = slot(std::integral_constant<int, (I + 1) % R>{});
        bf16x8(&nxc)[MT][4][64] = slot(std::integral_constant<int, (I + R - 1) % R>{});
        const bf16x8(&bq)[NTW][4] = fset(std::integral_constant<int, I % NB>{});
        bf16x8(&bn)[NTW][4] = fset(std::integral_constant<int, (I + NB - 1) % NB>{});
        const int wq = clampw(w + NB - 1), wc = clampw(w + R - 1);
#pragma unroll
        for (int g = 0; g < NG; g++) {
            if (g + 1 < NG) {
                read_group(a[(g + 1) & 1], cur, g + 1);
            } else {
                // the copies of w + 1 (issued R - 2 stages ago) are in
                wait_vmcnt_at_most<kInFlight>();
                block_barrier();
                read_group(a[0], nx1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < NM; i++) {
                mfma_one(a[g & 1], bq, g, i);
                if (g + 1 < NG) {
                    // fragments of w + NB - 1, spread over the first NG - 1 groups
                    constexpr int span = (NG - 1) * NM;
#pragma unroll
                    for (int l = 0; l < NQ; l++)
                        if (l * span / NQ == g * NM + i)
                            load_q1(bn, l, wq);
                } else {
#pragma unroll
                    for (int c = 0; c < CPW; c++)
                        if (c * NM / CPW == i)
                            copy_one(nxc, c, wc);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };
    // prologue: windows 0 .. R - 2 into the ring, fragments of windows
    // 0 .. NB - 2, group 0 of window 0
#pragma unroll
    for (int c = 0; c < CPW; c++) {
        copy_one(ring0, c, 0);
        copy_one(ring1, c, clampw(1));
        copy_one(ring2, c, clampw(2));
        if constexpr (R > 4) copy_one(ring3, c, clampw(3));
        if constexpr (R > 5) copy_one(ring4, c, clampw(4));
    }
#pragma unroll
    for (int l = 0; l < NQ; l++) {
        load_q1(b0, l, 0);
        if constexpr (NB > 2) load_q1(b1, l, clampw(1));
    }
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt_at_most<0>();
    __syncthreads();
    read_group(a[0], ring0, 0);
    // U stages per trip; the tail runs the last 0 .. U - 1 windows
    int w = 0;
    for (; w + U <= nwin; w += U)
        unrolled<U>([&](auto i_t) { stage(i_t, w + decltype(i_t)::value); });
    unrolled<U - 1>([&](auto i_t) {
        if (w + decltype(i_t)::value < nwin)
            stage(i_t, w + decltype(i_t)::value);
    });
    // no copy may still be writing LDS when the block ends
    wait_vmcnt_at_most<0>();

    // block keys, as in scan_mfma_kernel
    int32_t ex[NTW];
    float qs[NTW];
#pragma unroll
    for (int nt = 0; nt < NTW; nt++) {
        const int qb = (tg * NTW + nt) * 32 + r;
        ex[nt] = (exclude && qb < B) ? exclude[qb] : -1;
        qs[nt] = (FMT == kKeyBf16 || qb >= B) ? 1.f : qscale[qb];
    }
#pragma unroll
    for (int mt = 0; mt < MTW; mt++) {
        const int64_t rb = rb0 + rp * MTW + mt;
        int32_t pr[16];
        float ks[16];
        if (exclude)
            tile_rows_load(pr, prompt, rb * kRowBlock, h, n_valid);
        if constexpr (FMT == kKeyFp8)
            tile_rows_load(ks, kscale, rb * kRowBlock, h, n_valid);
#pragma unroll
        for (int nt = 0; nt < NTW; nt++) {
            const int qb = (tg * NTW + nt) * 32 + r;
            // the tile moves out of the accumulation registers here, one tile at a time
            floatx16 t = acc[mt][nt];
            asm volatile("" : "+v"(t));
            uint64_t best = 0;
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int64_t row = rb * kRowBlock + (e / 4) * 8 + h * 4 + e % 4;
                if (row < n_valid) {
                    float v = t[e];
                    if constexpr (FMT == kKeyFp8)
                        v = v * (ks[e] * qs[nt]);  // powers of two: exact, as the narrow scan scales it
                    if (ex[nt] >= 0 && pr[e] == ex[nt])
                        v = __uint_as_float(kNoScoreBits);
                    const uint64_t key = rank_key(v, (uint32_t)row);
                    best = key > best ? key : best;
                }
            }
            const uint64_t other = __shfl_xor(best, 32, kWave);
            best = other > best ? other : best;
            // streamed past the caches up to four query tiles (B = 128: 1.498
            // -> 1.460 ms); plain stores at 8 and 16 tiles, whose block keys
            // are 2-4x as many (B = 256 / 512: 2.11 / 3.63 ms against 2.18 /
            // 3.87 streamed)
            if (qb < B && h == 0 && rb * kRowBlock < n_valid) {
                if constexpr (NTW * WAVES / RS <= 4)
                    __builtin_nontemporal_store(best, &G[qb * g_ld + rb]);
                else
                    G[qb * g_ld + rb] = best;
            }
            __builtin_amdgcn_sched_barrier(0);  // one tile at a time: bounds the live registers
        }
    }
}

// ----------------------------------------------------------------- remainder of the B <= 64 scan
// Row blocks past the last whole generation of scan_mfma_kernel's waves are
// too few to keep HBM busy: each one's walk over the windows is bound by
// load latency, not bandwidth.  Here one workgroup takes one such row block:
// four copy waves stream its 4 KiB tiles into an LDS ring of TS chunks of TC
// windows (copy wave v moves the 1 KiB operand chunk v of every window, with
// buffer loads straight to LDS), so up to TS * TC windows are in flight, and
// NT compute waves, one per query tile, run the row block's MFMA sequence:
// the instructions of scan_mfma_kernel in the same order (windows in order,
// sub-steps in order), so every score is bit-identical to the main grid's
// and the rescore's.  The two kinds of waves run separate loops that meet at
// the same two barriers per chunk (chunk i in LDS; chunk i consumed, its slot
// free for chunk i + TS).  Query fragments go to registers TP windows ahead.
#ifndef OIL_TAIL_TC
#define OIL_TAIL_TC 8
#endif
#ifndef OIL_TAIL_TS
#define OIL_TAIL_TS 4
#endif
template <int NT, int FMT>
__global__ __launch_bounds__(64 * (NT + 4)) void scan_tail_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const bf16x8* __restrict__ qfrag, int32_t B, const int32_t* __restrict__ prompt,
    const int32_t* __restrict__ exclude, uint64_t* __restrict__ G, int64_t g_ld,
    const float* __restrict__ kscale, const float* __restrict__ qscale, int64_t rb_base)
{
    constexpr int TC = OIL_TAIL_TC, TS = OIL_TAIL_TS;
    constexpr int TP = TC - 1;  // fragment prefetch distance (windows); set of window w: w % TC
    static_assert(TC >= 2 && TS >= 2 && (TS - 1) * TC <= 63, "vmcnt range");
    __shared__ bf16x8 ring[TS][TC][4][64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform per wave
    const int h = lane >> 5, r = lane & 31;
    const int64_t rb = rb_base + blockIdx.x;
    const int nwin = ld / (FMT == kKeyBf16 ? kWindow : kWindowFp8);
    const int nch = (nwin + TC - 1) / TC;
    auto clampw = [&](int w) { return w < nwin ? w : nwin - 1; };

    if (wave >= NT) {
        // copy wave v: operand chunk v (1 KiB) of every window
        const int v = wave - NT;
        const char* src = (const char*)(keys + rb * rs) + v * 1024;
        const int64_t wbytes = ws * 2;
        const uint32_t loff = (uint32_t)lane * 16;
        auto issue = [&](int ch) {
            bf16x8(&buf)[TC][4][64] = ring[ch % TS];
#pragma unroll
            for (int c = 0; c < TC; c++) {
                const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
                    (void*)(src + clampw(ch * TC + c) * wbytes), (short)0, 1024, 0x00020000);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsrc, (void __attribute__((address_space(3)))*)&buf[c][v][0], 16, loff, 0, 0,
                    OIL_WIDE_KEY_CPOL);
            }
        };
        for (int ch = 0; ch < TS && ch < nch; ch++)
            issue(ch);
        for (int i = 0; i < nch; i++) {
            // this wave's copies of chunk i have landed: the copies of at
            // most TS - 1 later chunks may still be in flight
            const int later = nch - 1 - i < TS - 1 ? nch - 1 - i : TS - 1;
            unrolled<TS>([&](auto n_t) {
                constexpr int n = decltype(n_t)::value;
                if (later == n)
                    wait_vmcnt_at_most<n * TC>();
            });
            block_barrier();  // chunk i is in LDS
            block_barrier();  // chunk i has been read
            if (i + TS < nch)
                issue(i + TS);
        }
        return;
    }

    // compute wave nt: query tile nt
    const int nt = wave;
    const bf16x8* qf = qfrag + (int64_t)nt * 4 * 64 + lane;
    auto load_frag = [&](bf16x8 (&b)[4], int w) {
#pragma unroll
        for (int s = 0; s < 4; s++)
            b[s] = qf[(((int64_t)w * NT) * 4 + s) * 64];
    };
    bf16x8 fb[TC][4];
#pragma unroll
    for (int p = 0; p < TP; p++)
        load_frag(fb[p], clampw(p));
    floatx16 acc = floatx16{};
    // A operands: two register sets; window c's in set c % 2, read while
    // window c - 1's MFMAs run (a chunk's first window: after its barrier)
    bf16x8 a0[4], a1[4];
    auto aset = [&](auto k_t) -> bf16x8(&)[4] {
        if constexpr (decltype(k_t)::value == 0) return a0;
        else return a1;
    };
    auto read_a = [&](bf16x8 (&a)[4], const bf16x8(&buf)[TC][4][64], int c) {
#pragma unroll
        for (int s = 0; s < 4; s++)
            a[s] = buf[c][s][lane];
    };
    // window c of chunk i: the fragments of window w + TP requested, the A
    // operands of window c + 1 read, then window c's MFMAs (the scheduling
    // barriers keep each window's loads and MFMAs in that order)
    auto window = [&](const bf16x8(&buf)[TC][4][64], auto c_t, int w) {
        constexpr int c = decltype(c_t)::value;
        load_frag(fb[(c + TP) % TC], clampw(w + TP));
        if constexpr (c + 1 < TC)
            read_a(aset(std::integral_constant<int, (c + 1) % 2>{}), buf, c + 1);
        __builtin_amdgcn_sched_barrier(0x0006);
        const bf16x8(&a)[4] = aset(std::integral_constant<int, c % 2>{});
        if constexpr (FMT == kKeyFp8) {
            acc = mfma_pair_fp8(a[0], a[1], fb[c][0], fb[c][1], acc);
            acc = mfma_pair_fp8(a[2], a[3], fb[c][2], fb[c][3], acc);
        } else {
#pragma unroll
            for (int s = 0; s < 4; s++)
                acc = mfma_step(a[s], fb[c][s], acc);
        }
        __builtin_amdgcn_sched_barrier(0x0006);
    };
    const int nfull = nwin / TC;
    for (int i = 0; i < nfull; i++) {
        block_barrier();  // chunk i is in LDS
        const bf16x8(&buf)[TC][4][64] = ring[i % TS];
        read_a(a0, buf, 0);
        unrolled<TC>([&](auto c_t) { window(buf, c_t, i * TC + decltype(c_t)::value); });
        block_barrier();  // chunk i has been read
    }
    if (nfull < nch) {  // the last, partial chunk
        block_barrier();
        const bf16x8(&buf)[TC][4][64] = ring[nfull % TS];
        read_a(a0, buf, 0);
        unrolled<TC>([&](auto c_t) {
            const int w = nfull * TC + decltype(c_t)::value;
            if (w < nwin)
                window(buf, c_t, w);
        });
        block_barrier();
    }

    // block keys, as in scan_mfma_kernel
    const int qb = nt * 32 + r;
    const bool qlive = qb < B;
    const int32_t ex = (exclude && qlive) ? exclude[qb] : -1;
    const float qs = (FMT == kKeyBf16 || !qlive) ? 1.f : qscale[qb];
    int32_t pr[16];
    float ks[16];
    if (exclude)
        tile_rows_load(pr, prompt, rb * kRowBlock, h, n_valid);
    if constexpr (FMT == kKeyFp8)
        tile_rows_load(ks, kscale, rb * kRowBlock, h, n_valid);
    uint64_t best = 0;
#pragma unroll
    for (int e = 0; e < 16; e++) {
        const int64_t row = rb * kRowBlock + (e / 4) * 8 + h * 4 + e % 4;
        if (row < n_valid) {
            float v = acc[e];
            if constexpr (FMT == kKeyFp8)
                v = v * (ks[e] * qs);  // powers of two: exact
            if (ex >= 0 && pr[e] == ex)
                v = __uint_as_float(kNoScoreBits);
            const uint64_t key = rank_key(v, (uint32_t)row);
            best = key > best ? key : best;
        }
    }
    const uint64_t other = __shfl_xor(best, 32, kWave);
    best = other > best ? other : best;
    if (qlive && h == 0)
        __builtin_nontemporal_store(best, &G[qb * g_ld + rb]);
}

// ----------------------------------------------------------------- rescore the chosen blocks
// One wave per (chosen block slot, query).  The block comes from its best key
// (0: no block, the slot's scores are "no position").  Scores land in
// SC[(query * k + slot) * 32 + row in block].

// MFMA path: the same v_mfma_f32_32x32x16_bf16 sequence as the scan (windows
// in order, sub-steps in order, starting from zero) on the block's tile and
// the query's 32-query fragment tile, so element (row, query) is bit-identical
// to the scan's; the wave keeps the query's column.
template <int PF, int FMT>
__global__ __launch_bounds__(64) void rescore_mfma_kernel(
    const uint16_t* __restrict__ keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
    const bf16x8* __restrict__ qfrag, int n_qtiles, const uint64_t* __restrict__ blocks, int k,
    const int32_t* __restrict__ prompt, const int32_t* __restrict__ exclude, float* __restrict__ SC,
    const float* __restrict__ kscale, const float* __restrict__ qscale)
{
    constexpr int NS = PF + 1;
    const int slot = blockIdx.x, qb = blockIdx.y, lane = threadIdx.x;
    const int h = lane >> 5, r = lane & 31;
    float* out = SC + ((int64_t)qb * k + slot) * kRowBlock;
    const uint64_t bk = blocks[(int64_t)qb * k + slot];
    const int64_t rb = key_pos(bk) / kRowBlock;
    // no block (or, defensively, one past the pool: nothing is read there)
    if (bk == 0 || rb * kRowBlock >= n_valid) {
        if (lane < kRowBlock)
            out[lane] = __uint_as_float(kNoScoreBits);
        return;
    }
    const int t = qb >> 5, n = qb & 31;
    const int nwin = ld / (FMT == kKeyBf16 ? kWindow : kWindowFp8);
    const int64_t ws8 = ws / 8;
    const bf16x8* tile = (const bf16x8*)(keys + rb * rs) + lane;
    // Every column of the B operand gets this query's fragment (lane h * 32 + c
    // reads lane h * 32 + n's): an MFMA output element depends only on its own
    // row and column, so column n comes out as in the scan, and the wave reads
    // 32 bytes of query per sub-step instead of the whole query tile's 1 KiB.
    const bf16x8* qf = qfrag + ((lane & 32) | n);
    floatx16 acc = floatx16{};
    bf16x8 a[NS][4], b[NS][4];
    auto load = [&](int stage, int w) {
#pragma unroll
        for (int s = 0; s < 4; s++) {
            a[stage][s] = __builtin_nontemporal_load(tile + w * ws8 + s * 64);
            b[stage][s] = qf[(((int64_t)w * n_qtiles + t) * 4 + s) * 64];
        }
    };
#pragma unroll
    for (int p = 0; p < PF; p++)
        load(p, p < nwin ? p : nwin - 1);
    const int nloop = (nwin + NS - 1) / NS * NS;
    for (int w0 = 0; w0 < nloop; w0 += NS) {
#pragma unroll
        for (int u = 0; u < NS; u++) {
            const int wl = w0 + u + PF < nwin ? w0 + u + PF : nwin - 1;
            load((u + PF) % NS, wl);
            if (w0 + u < nwin) {
                if constexpr (FMT == kKeyFp8) {
                    acc = mfma_pair_fp8(a[u][0], a[u][1], b[u][0], b[u][1], acc);
                    acc = mfma_pair_fp8(a[u][2], a[u][3], b[u][2], b[u][3], acc);
                } else {
#pragma unroll
                    for (int s = 0; s < 4; s++)
                        acc = mfma_step(a[u][s], b[u][s], acc);
                }
            }
        }
    }
    if (r != n)
        return;
    const int32_t ex = exclude ? exclude[qb] : -1;
    float ks[16];
    int32_t pr[16];
    if constexpr (FMT == kKeyFp8)
        tile_rows_load(ks, kscale, rb * kRowBlock, h, n_valid);
    if (ex >= 0)
        tile_rows_load(pr, prompt, rb * kRowBlock, h, n_valid);
    const float qs = FMT == kKeyFp8 ? qscale[qb] : 1.f;
#pragma unroll
    for (int e = 0; e < 16; e++) {
        const int rr = (e / 4) * 8 + h * 4 + e % 4;
        const int64_t row = rb * kRowBlock + rr;
        float v = acc[e];
        if constexpr (FMT == kKeyFp8)
            v = v * (ks[e] * qs);  // as the scan scales it
        if (row >= n_valid || (ex >= 0 && pr[e] == ex))
            v = __uint_as_float(kNoScoreBits);
        out[rr] = v;
    }
}

// ----------------------------------------------------------------- launchers
// The GEMV keeps all queries of the call in LDS (at most 64 KiB).
int scan_uses_mfma(int32_t B, int32_t ld) { return B > 4 || (int64_t)B * ld * 2 > 65536; }

int scan_query_tiles(int32_t B) { return (B + 31) / 32; }

// Where a scan's kernels go: the stream, and two events (or null) that
// hipExtLaunchKernel binds to the scan's first and last kernels, for timing.
// Either way of taking events (bound, or recorded between kernels) delays
// the kernel after each event by a few microseconds, so callers time a
// sample of the scans.
struct ScanLaunch {
    hipStream_t stream;
    hipEvent_t start, stop;
};

// Launch one 256-thread scan kernel; first / last say whether it is the
// scan's first / last kernel (which carry the events).
template <class K, class... A>
static void dispatch_n(const ScanLaunch& sl, bool first, bool last, K kernel, dim3 grid, dim3 block, size_t lds,
                       A... args)
{
    hipEvent_t s = first ? sl.start : nullptr, e = last ? sl.stop : nullptr;
    if (s || e)
        hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, sl.stream, s, e, 0u, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, sl.stream, args...);
}
template <class K, class... A>
static void dispatch(const ScanLaunch& sl, bool first, bool last, K kernel, dim3 grid, size_t lds, A... args)
{
    dispatch_n(sl, first, last, kernel, grid, dim3(256), lds, args...);
}

template <int NB>
static void launch_gemv(dim3 g, size_t lds, const ScanLaunch& sl, const uint16_t* keys, int32_t ld,
                        int64_t rs, int64_t ws, int64_t n_valid, const uint16_t* q,
                        const int32_t* prompt, const int32_t* exclude, uint64_t* G, int64_t g_ld, float* FS,
                        int64_t fs_ld)
{
    dispatch(sl, true, true, scan_gemv_kernel<NB, 3>, g, lds, keys, ld, rs, ws, n_valid, q, prompt, exclude, G,
             g_ld, FS, fs_ld);
}

static bool nwin_even(int32_t ld, int fmt) { return (ld / (fmt == kKeyBf16 ? kWindow : kWindowFp8)) % 2 == 0; }

// Compute units of the current device (cached per device).
static int device_cus()
{
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 256;
    if (cus[dev] == 0) {
        int n = 0;
        cus[dev] = (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
                       ? n
                       : 256;
    }
    return cus[dev];
}

// The MFMA scan for B <= 64.  Each wave walks every key window of its MT row
// blocks, so a wave lives as long as the whole scan when the chip is full.
// Row blocks that fill whole generations of waves (all the SIMDs can hold)
// go to the main grid; a small remainder would leave a few waves walking every window
// nearly alone at the end (latency-bound, about 2-3 us per window pair), so
// it goes to a second launch with one row block per wave and TPF windows in
// flight.  Every row block's MFMA sequence is the same in both launches.
template <int MT, int NT, int PF, int TPF, int FMT>
static void launch_narrow(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid, int64_t n_rb,
                          const bf16x8* qf, int32_t B, const int32_t* prompt, const int32_t* exclude,
                          uint64_t* G, int64_t g_ld, const float* kscale, const float* qscale, const ScanLaunch& sl)
{
    constexpr int kWavesPerSimd = NT == 1 ? 2 : 1;  // what the kernels' register use allows
    const int64_t gen = (int64_t)device_cus() * 4 * kWavesPerSimd * MT;
    // Measured on 1M x 4096 (B = 32, four generations): a remainder of 1-15
    // row blocks costs the main grid 0-30 us (its waves start while the last
    // generation runs), the second launch 14-30 us; from 16 on the main grid
    // pays 30-75 us, the second launch 23-34 us.  With one generation
    // (262,144 x 5,120, B = 16) the remainder's waves start only when the
    // generation ends: 2 / 7 / 15 row blocks cost the main grid 16 / 37 /
    // 87 us, the second launch 28 / 41 / 41 us.
    // scan_tail_kernel (one workgroup per row block, a deep LDS ring) takes
    // such a remainder when it holds at most one row block per compute unit:
    // about 12 us at 1M x 4096 (B = 32) whatever the count.  Past two or more
    // generations, fewer than 16 row blocks stay in the main grid (measured
    // there: about 2 us for 8-15 of them).
    constexpr int64_t kTailMin = 16, kTailMinOneGen = 8;
    int64_t n_main = n_rb, n_tail = 0;
    bool lds_tail = false;
    if (n_rb > gen) {
        const int64_t rem = n_rb % gen;
        const int64_t tail_min = n_rb < 2 * gen ? kTailMinOneGen : kTailMin;
        if (OIL_TAIL_LDS && rem >= (n_rb < 2 * gen ? 1 : kTailMin) && rem <= device_cus()) {
            n_main = n_rb - rem;
            n_tail = rem;
            lds_tail = true;
        } else if (rem >= tail_min && rem <= gen / 4) {
            n_main = n_rb - rem;
            n_tail = rem;
        }
    }
    if constexpr (NT == 1 && PF == 1 && (FMT == kKeyBf16 || OIL_SCAN_PERSIST_FP8)) {
        // Two or more whole rounds of groups (and a last round at least half
        // full): the persistent kernel, plus the remainder kernel for up to one
        // row block per compute unit past its groups
        // (the bench pool, 1M plus 8-15 row blocks: 1.378 -> 1.363 ms per
        // step).  With two query tiles the persistent form measured slower
        // (B = 64: 1.95 against 1.30 ms); with fp8 keys it gains at exactly 1M
        // (B = 32: 0.675 -> 0.665 ms) but loses on the bench pool, whose
        // remainder then costs a launch (0.7315 -> 0.7363 ms per step).
        const int64_t grp = 4 * MT;
        const int64_t per_round = (int64_t)device_cus() * kWavesPerSimd;  // workgroups the chip holds
        const int64_t full = n_rb / grp, rounds = full / per_round, part = full % per_round;
        // whole rounds, or all whole groups when the last round is at least half full
        int64_t n_groups = rounds * per_round;
        if (OIL_SCAN_PERSIST_PART && 2 * part >= per_round)
            n_groups = full;
        const int64_t rem = n_rb - n_groups * grp;
        if (OIL_SCAN_PERSIST && nwin_even(ld, FMT) && rounds >= 2 && rem <= device_cus()) {
            dispatch(sl, true, rem == 0, scan_mfma_persist_kernel<MT, NT, FMT>, dim3((unsigned)per_round), 0, keys,
                     ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale, n_groups);
            if (rem > 0)
                dispatch_n(sl, false, true, scan_tail_kernel<NT, FMT>, dim3((unsigned)rem), dim3(64 * (NT + 4)), 0,
                           keys, ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale,
                           n_groups * grp);
            return;
        }
    }
    dispatch(sl, true, n_tail == 0, scan_mfma_kernel<MT, NT, PF, FMT>,
             dim3((unsigned)((n_main + 4 * MT - 1) / (4 * MT))), 0, keys, ld, rs, ws, n_valid, qf, B, prompt,
             exclude, G, g_ld, kscale, qscale, (int64_t)0);
    if (lds_tail)
        dispatch_n(sl, false, true, scan_tail_kernel<NT, FMT>, dim3((unsigned)n_tail), dim3(64 * (NT + 4)), 0,
                   keys, ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale, n_main);
    else if (n_tail > 0)
        dispatch(sl, false, true, scan_mfma_kernel<1, NT, TPF, FMT>, dim3((unsigned)((n_tail + 3) / 4)), 0, keys,
                 ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale, n_main);
}

// The wide scan (64 < B <= 512), either key format: one configuration per
// class of batches (up to 4, 8 and 16 query tiles), (MT, R, NB, WAVES, WPE,
// RS): row blocks per workgroup, key windows in the LDS ring, fragment
// register sets, waves per workgroup, the waves per SIMD the registers must
// allow, and the waves that split a tile's row blocks.
template <int MT, int R, int NB, int WAVES, int WPE, int RS, int TILES, int FMT>
static void launch_wide_cfg(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
                            int64_t n_rb, const bf16x8* qf, int32_t B, const int32_t* prompt,
                            const int32_t* exclude, uint64_t* G, int64_t g_ld, const float* kscale,
                            const float* qscale, const ScanLaunch& sl)
{
    constexpr int NTW = TILES * RS / WAVES;
    static_assert(NTW * WAVES == TILES * RS, "query tiles per wave");
    const dim3 grid((unsigned)((n_rb + MT - 1) / MT)), block(64 * WAVES);
    // a batch that fills the class's tiles runs without the skip branches
    if (scan_query_tiles(B) == TILES)
        dispatch_n(sl, true, true, scan_mfma_wide_kernel<MT, NTW, R, NB, WAVES, WPE, FMT, RS, 0>, grid, block, 0, keys,
                   ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale);
    else
        dispatch_n(sl, true, true, scan_mfma_wide_kernel<MT, NTW, R, NB, WAVES, WPE, FMT, RS, 1>, grid, block, 0, keys,
                   ld, rs, ws, n_valid, qf, B, prompt, exclude, G, g_ld, kscale, qscale);
}

// Configurations (MT, R, NB, WAVES, WPE, RS) per class, measured on
// the 1M x 4096 pool (scan ms at B = 128 / 256 / 512; before: 1.71 / 2.39 /
// 4.43 with 4 row blocks, 4 waves and direct copies issued at the top of each
// window): bf16 8 row blocks, 8 waves (two per SIMD), each 4 row blocks of
// one tile: 1.49-1.51 (4 waves of 8 row blocks, keys through registers,
// 1.58-1.65; a five-window ring 1.52; keys through registers 1.54; 4 row
// splits 1.62; 4 row blocks 1.77); 8 row blocks and 8 waves of 8 row blocks
// each: 2.05-2.17 (row split 2.05-2.06; 4 row blocks and 4 waves 2.19-2.21,
// with three fragment sets 2.35); 4 row blocks and 8 waves (two per SIMD, 2
// query tiles each): 3.56-3.69 (4 waves of 4 tiles 3.73-3.82; a five-window
// ring 4.0; row splits need more than 256 registers).  fp8 (windows of 128
// columns): 0.88 / 1.29-1.35 / 2.18-2.22 (before: 0.97 / 1.31 / 2.56; 4 row
// blocks of 4 waves at B <= 128: 0.95).
#ifndef OIL_WIDE_C1
#define OIL_WIDE_C1 8, 4, 2, 8, 2, 2
#endif
#ifndef OIL_WIDE_C2
#define OIL_WIDE_C2 8, 4, 2, 8, 1, 1
#endif
#ifndef OIL_WIDE_C4
#define OIL_WIDE_C4 4, 4, 2, 8, 2, 1
#endif
#ifndef OIL_WIDE_F1
#define OIL_WIDE_F1 8, 4, 2, 8, 2, 2
#endif
#ifndef OIL_WIDE_F2
#define OIL_WIDE_F2 4, 4, 2, 8, 2, 1
#endif
#ifndef OIL_WIDE_F4
#define OIL_WIDE_F4 4, 4, 2, 4, 1, 1
#endif

template <int FMT>
static void launch_wide(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid, int64_t n_rb,
                        const bf16x8* qf, int32_t B, const int32_t* prompt, const int32_t* exclude, uint64_t* G,
                        int64_t g_ld, const float* kscale, const float* qscale, const ScanLaunch& sl)
{
    const int n_qt = scan_query_tiles(B);
#define OIL_WIDE_ARGS keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude, G, g_ld, kscale, qscale, sl
    if constexpr (FMT == kKeyBf16) {
        if (n_qt <= 4) launch_wide_cfg<OIL_WIDE_C1, 4, FMT>(OIL_WIDE_ARGS);
        else if (n_qt <= 8) launch_wide_cfg<OIL_WIDE_C2, 8, FMT>(OIL_WIDE_ARGS);
        else launch_wide_cfg<OIL_WIDE_C4, 16, FMT>(OIL_WIDE_ARGS);
    } else {
        if (n_qt <= 4) launch_wide_cfg<OIL_WIDE_F1, 4, FMT>(OIL_WIDE_ARGS);
        else if (n_qt <= 8) launch_wide_cfg<OIL_WIDE_F2, 8, FMT>(OIL_WIDE_ARGS);
        else launch_wide_cfg<OIL_WIDE_F4, 16, FMT>(OIL_WIDE_ARGS);
    }
#undef OIL_WIDE_ARGS
}

hipError_t launch_scan(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
                       const void* qbuf, int32_t B, const int32_t* prompt, const int32_t* exclude,
                       uint64_t* G, int64_t g_ld, hipStream_t stream, int fmt, const float* kscale,
                       const float* qscale, hipEvent_t ev_start, hipEvent_t ev_stop, float* FS, int64_t fs_ld)
{
    if (n_valid <= 0)
        return hipSuccess;
    const ScanLaunch sl{stream, ev_start, ev_stop};
    const int64_t n_rb = (n_valid + kRowBlock - 1) / kRowBlock;
    if (fmt == kKeyFp8) {
        constexpr int MT = OIL_FP8_MT, MT2 = OIL_FP8_MT2, PF = OIL_FP8_PF;
        const bf16x8* qf = (const bf16x8*)qbuf;
        if (B > 64)
            launch_wide<kKeyFp8>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude, G, g_ld, kscale, qscale,
                                 sl);
        else if (scan_query_tiles(B) == 1)
            launch_narrow<MT, 1, PF, OIL_TAIL_PF1, kKeyFp8>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude,
                                                            G, g_ld, kscale, qscale, sl);
        else
            launch_narrow<MT2, 2, PF, OIL_TAIL_PF2, kKeyFp8>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude,
                                                             G, g_ld, kscale, qscale, sl);
        return hipGetLastError();
    }
    if (!scan_uses_mfma(B, ld) && FS) {  // the GEMV scan only where it writes every score
        const dim3 g((unsigned)((n_rb + 3) / 4));
        const size_t lds = (size_t)B * ld * sizeof(uint16_t);
        const uint16_t* q = (const uint16_t*)qbuf;
        switch (B) {
        case 1: launch_gemv<1>(g, lds, sl, keys, ld, rs, ws, n_valid, q, prompt, exclude, G, g_ld, FS, fs_ld); break;
        case 2: launch_gemv<2>(g, lds, sl, keys, ld, rs, ws, n_valid, q, prompt, exclude, G, g_ld, FS, fs_ld); break;
        case 3: launch_gemv<3>(g, lds, sl, keys, ld, rs, ws, n_valid, q, prompt, exclude, G, g_ld, FS, fs_ld); break;
        default: launch_gemv<4>(g, lds, sl, keys, ld, rs, ws, n_valid, q, prompt, exclude, G, g_ld, FS, fs_ld); break;
        }
        return hipGetLastError();
    }
    const bf16x8* qf = (const bf16x8*)qbuf;
    if (B > 64) {
        launch_wide<kKeyBf16>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude, G, g_ld, nullptr, nullptr,
                              sl);
        return hipGetLastError();
    }
    constexpr int MT = OIL_BF16_MT, MT2 = OIL_BF16_MT2, PF = OIL_BF16_PF;
    if (scan_query_tiles(B) == 1)
        launch_narrow<MT, 1, PF, OIL_TAIL_PF1, kKeyBf16>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude, G,
                                                         g_ld, nullptr, nullptr, sl);
    else
        launch_narrow<MT2, 2, PF, OIL_TAIL_PF2, kKeyBf16>(keys, ld, rs, ws, n_valid, n_rb, qf, B, prompt, exclude, G,
                                                          g_ld, nullptr, nullptr, sl);
    return hipGetLastError();
}

hipError_t launch_rescore(const uint16_t* keys, int32_t ld, int64_t rs, int64_t ws, int64_t n_valid,
                          const void* qbuf, int32_t B, const uint64_t* blocks, int32_t k,
                          const int32_t* prompt, const int32_t* exclude, float* SC, hipStream_t stream,
                          int fmt, const float* kscale, const float* qscale)
{
    const dim3 g((unsigned)k, (unsigned)B);
    if (fmt == kKeyFp8)
        hipLaunchKernelGGL((rescore_mfma_kernel<OIL_RESCORE_PF, kKeyFp8>), g, dim3(64), 0, stream, keys, ld, rs, ws, n_valid,
                           (const bf16x8*)qbuf, scan_query_tiles(B), blocks, k, prompt, exclude, SC, kscale,
                           qscale);
    else
        hipLaunchKernelGGL((rescore_mfma_kernel<OIL_RESCORE_PF, kKeyBf16>), g, dim3(64), 0, stream, keys, ld, rs, ws, n_valid,
                           (const bf16x8*)qbuf, scan_query_tiles(B), blocks, k, prompt, exclude, SC, nullptr,
                           nullptr);
    return hipGetLastError();
}

}  // namespace oil
