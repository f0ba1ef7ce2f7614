// gfx950 kernels and C ABI of the automated mixed-bit allocation of ShiftAddLLM
// (Sec. 4.3): the criterion of Eq. 3 for one layer, the per-bit least-squares
// fits, and the integer program of Eq. 4.
//
//   IS = W / diag(cholesky(H^-1)),  H = X X^T + damp * mean(diag(X X^T)) I,
//   C  = ||IS||_F * STD(IS)^2
//
// computed as: the Gram matrix X X^T of fp16 calibration activations on the
// matrix cores (v_mfma_f32_16x16x32_f16, fp32 accumulation; only the lower
// triangle of tiles); the damped matrix in fp64 with rows and columns in reverse
// order; a blocked fp64 Cholesky of it, because the diagonal of the Cholesky
// factor of H^-1 is, in reverse order, the reciprocal of the diagonal of the
// Cholesky factor of the reversed H (no inverse is formed); and fp64 sums of IS
// and IS^2 in a fixed order.  Eq. 4 is a multiple-choice knapsack over integer
// bit totals, solved exactly on the host.
#include <hip/hip_runtime.h>

#include <mutex>

#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <type_traits>
#include <vector>

#include "shiftadd.h"

namespace {

// ---------------------------------------------------------------- Gram matrix

// Lower-triangular tile (ti, tj), ti >= tj, of linear block index b.
__device__ inline void lower_tile(int b, int& ti, int& tj) {
    int t = (int)((sqrtf(8.0f * b + 1.0f) - 1.0f) * 0.5f);
    while ((t + 1) * (t + 2) / 2 <= b) ++t;
    while (t * (t + 1) / 2 > b) --t;
    ti = t;
    tj = b - t * (t + 1) / 2;
}

constexpr int kGT = 128;       // output tile: 128 x 128
constexpr int kGK = 32;        // calibration columns per stage
// LDS row stride in halves (80 bytes): 16-byte aligned rows whose 16-byte
// operand reads by 16 consecutive rows cover all 64 banks once
constexpr int kGPad = kGK + 8;
constexpr int kGBuf = kGT * kGPad;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

// Tile (ti, tj), ti >= tj, of H = X X^T for X fp16 [K][T] row-major.  Four
// waves, each a 64 x 64 quarter (4 x 4 blocks of 16 x 16, 16 accumulators of
// four floats).  The two 128 x 32 slices of X of a stage are double-buffered
// in LDS; the next stage's slices are loaded into registers while the current
// one is multiplied, so one barrier per stage suffices.
// Operand layout of v_mfma_f32_16x16x32_f16 (gfx950; twice the products per
// instruction of the 16x16x16 form at about the same issue cost, measured):
// lane l holds row (l mod 16) of A and column (l mod 16) of B at
// k = 8 (l / 16) .. 8 (l / 16) + 7; the result holds rows 4 (l / 16) .. + 3 of
// column (l mod 16).
__global__ __launch_bounds__(256) void k_gram_f16(const uint16_t* __restrict__ x, int K, int T,
                                                  float* __restrict__ H) {
    __shared__ uint16_t sa[2 * kGBuf];
    __shared__ uint16_t sb[2 * kGBuf];
    int ti, tj;
    lower_tile((int)blockIdx.x, ti, tj);
    const int i0 = ti * kGT, j0 = tj * kGT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wi = (wave >> 1) * 64, wj = (wave & 1) * 64;
    // staging: thread -> rows lr and lr + 64, 8 halves at column lc
    const int lr = tid >> 2, lc = (tid & 3) * 8;
    const uint16_t* pa = x + (int64_t)(i0 + lr) * T + lc;
    const uint16_t* pb = x + (int64_t)(j0 + lr) * T + lc;
    const int64_t half = (int64_t)64 * T;
    float4v acc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = float4v{0.f, 0.f, 0.f, 0.f};
    const int r16 = lane & 15, kq = (lane >> 4) * 8;

    uint4 ra0 = *reinterpret_cast<const uint4*>(pa);
    uint4 ra1 = *reinterpret_cast<const uint4*>(pa + half);
    uint4 rb0 = *reinterpret_cast<const uint4*>(pb);
    uint4 rb1 = *reinterpret_cast<const uint4*>(pb + half);
    auto stage_store = [&](int buf) {
        uint16_t* A = sa + buf * kGBuf;
        uint16_t* Bm = sb + buf * kGBuf;
        *reinterpret_cast<uint4*>(A + lr * kGPad + lc) = ra0;
        *reinterpret_cast<uint4*>(A + (lr + 64) * kGPad + lc) = ra1;
        *reinterpret_cast<uint4*>(Bm + lr * kGPad + lc) = rb0;
        *reinterpret_cast<uint4*>(Bm + (lr + 64) * kGPad + lc) = rb1;
    };
    stage_store(0);
    __syncthreads();
    const int stages = T / kGK;
    for (int st = 0; st < stages; ++st) {
        const int buf = st & 1;
        if (st + 1 < stages) {
            const int t1 = (st + 1) * kGK;
            ra0 = *reinterpret_cast<const uint4*>(pa + t1);
            ra1 = *reinterpret_cast<const uint4*>(pa + half + t1);
            rb0 = *reinterpret_cast<const uint4*>(pb + t1);
            rb1 = *reinterpret_cast<const uint4*>(pb + half + t1);
        }
        const uint16_t* A = sa + buf * kGBuf;
        const uint16_t* Bm = sb + buf * kGBuf;
#pragma unroll
        for (int ks = 0; ks < kGK; ks += 32) {
            half8 av[4], bv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                av[u] = __builtin_bit_cast(half8, *reinterpret_cast<const uint4*>(
                                                      A + (wi + 16 * u + r16) * kGPad + ks + kq));
                bv[u] = __builtin_bit_cast(half8, *reinterpret_cast<const uint4*>(
                                                      Bm + (wj + 16 * u + r16) * kGPad + ks + kq));
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    acc[u][v] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[u], bv[v], acc[u][v], 0, 0, 0);
        }
        if (st + 1 < stages) stage_store(buf ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = i0 + wi + 16 * u + (lane >> 4) * 4 + e;
                const int j = j0 + wj + 16 * v + r16;
                H[(int64_t)i * K + j] = acc[u][v][e];
                if (ti != tj) H[(int64_t)j * K + i] = acc[u][v][e];
            }
}

// ---------------------------------------------------------------- Gram matrix, large shapes
//
// For many calibration tokens the per-tile kernel above is bound by its own
// operand traffic (a 128 x 128 tile reads 256 rows of X per 32 columns) and by
// one wave per SIMD stalling on each stage.  The large-shape path works on
// 256-row super-panels of X:
//   * an off-diagonal 256 x 256 region of H (super-rows a > b) is split into
//     two halves of the calibration columns, one workgroup each; the two fp32
//     partials are added onto zero, which gives the same bits in either order;
//   * a diagonal region (a, a) is one workgroup over all columns computing 8 of
//     the 10 lower-triangle 64 x 64 quadrants; the other two, (3,2) and (3,3),
//     are split over pieces of the columns (k_gram_rest) whose partials are
//     kept in strictly-upper tiles of H and summed in piece order
//     (k_gram_reduce);
//   * finally the lower triangle is mirrored (k_gram_mirror).
// With K = 4096 that is 256 equal workgroups, one per compute unit.  Operands
// travel global -> LDS directly (16 bytes per lane, no register staging) into
// a ring of four 32-column stages, two stages ahead of the one multiplied.

constexpr int kGS = 256;       // super-panel rows
constexpr int kGS2 = 32;       // calibration columns per stage (64-byte rows, 4 chunks)
constexpr int kGRing = 4;      // LDS ring depth
constexpr int kGPieces = 16;   // column pieces of each leftover quadrant pair

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte chunk c of LDS row r sits at chunk c ^ ((r >> 1) & 3): the operand
// reads (16 consecutive rows, one chunk) and the 1 KB DMA blocks are both free
// of bank conflicts (measured).
__device__ inline int gswz(int row, int chunk) { return chunk ^ ((row >> 1) & 3); }

__device__ inline uint32_t lds_address(const void* p) {
    return (uint32_t)(uintptr_t)((__attribute__((address_space(3))) const char*)(const char*)p);
}
// One global -> LDS load of 16 bytes per lane: lane l's bytes land at lds + 16 l.
// M0 carries the LDS address; nothing else in these kernels uses M0.  The
// compiler does not see these loads, so every wait on them is explicit.
__device__ inline void dma16(const uint16_t* g, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds) : "memory");
}
template <int N>
__device__ inline void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ inline void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Work item li -> region: first the first halves of all off-diagonal regions
// (a > b), then the diagonal regions, then the second halves.  Off-diagonal
// regions are listed in blocks of 4 super-rows x 8 super-columns, so the 32
// consecutive items one XCD receives share few panels of X at one position in
// the calibration columns (its L2 serves them all).
__device__ inline void gram_offdiag(int idx, int np, int& a, int& b) {
    for (int a0 = 0; a0 < np; a0 += 4) {
        const int a1 = min(np, a0 + 4);
        for (int b0 = 0; b0 < a1 - 1; b0 += 8) {
            const int b1 = b0 + 8;
            int cnt = 0;
            for (int x = a0; x < a1; ++x) cnt += max(0, min(b1, x) - b0);
            if (idx < cnt) {
                for (int x = a0; x < a1; ++x) {
                    const int k = max(0, min(b1, x) - b0);
                    if (idx < k) {
                        a = x;
                        b = b0 + idx;
                        return;
                    }
                    idx -= k;
                }
            }
            idx -= cnt;
        }
    }
    a = b = 0;
}
__device__ inline void gram_region_of(int li, int np, int& a, int& b, int& half, bool& diag) {
    const int n_off = np * (np - 1) / 2;
    diag = li >= n_off && li < n_off + np;
    half = li >= n_off + np ? 1 : 0;
    if (diag) {
        a = b = li - n_off;
        return;
    }
    gram_offdiag(half ? li - n_off - np : li, np, a, b);
}

// Eight waves.  Off-diagonal: wave w owns rows 128 (w >> 2) .. + 127 of the
// A panel against rows 64 (w & 3) .. + 63 of the B panel (8 x 4 blocks of
// 16 x 16).  Diagonal: wave w owns quadrant w of (0,0) (1,0) (1,1) (2,0)
// (2,1) (2,2) (3,0) (3,1), both operands from the one panel.
template <bool DIAG>
__device__ inline void gram_region(const uint16_t* __restrict__ x, int K, int T, float* __restrict__ H,
                                   int a, int bsr, int half, uint16_t* const* Ar, uint16_t* const* Br) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r16 = lane & 15, q = lane >> 4;
    const int arow0 = kGS * a, brow0 = kGS * bsr;
    constexpr int NDMA = DIAG ? 2 : 4;   // loads per wave per stage
    const int S = T / kGS2;
    const int sb = DIAG ? 0 : (half ? S / 2 : 0), se = DIAG ? S : (half ? S : S / 2);
    // DMA rows of this wave: 32 w + 16 i + (lane >> 2), i < 2 (one 1 KB block per
    // instruction); the swizzled chunk does not depend on i.  Rows past K read row K-1
    // (their products only reach entries of H that are not written).
    const int lrow = 32 * w + (lane >> 2);
    const int chunk = gswz(lrow, lane & 3);
    const uint16_t* pa0 = x + (int64_t)min(arow0 + lrow, K - 1) * T + 8 * chunk;
    const uint16_t* pa1 = x + (int64_t)min(arow0 + lrow + 16, K - 1) * T + 8 * chunk;
    const uint16_t* pb0 = x + (int64_t)min(brow0 + lrow, K - 1) * T + 8 * chunk;
    const uint16_t* pb1 = x + (int64_t)min(brow0 + lrow + 16, K - 1) * T + 8 * chunk;
    const int wu = __builtin_amdgcn_readfirstlane(w);
    auto issue = [&](int st, int slot) __attribute__((always_inline)) {
        const int t0 = st * kGS2;
        const uint32_t la = lds_address(Ar[slot]) + (uint32_t)(32 * wu) * (kGS2 * 2);
        dma16(pa0 + t0, la);
        dma16(pa1 + t0, la + 16 * (kGS2 * 2));
        if (!DIAG) {
            const uint32_t lb = lds_address(Br[slot]) + (uint32_t)(32 * wu) * (kGS2 * 2);
            dma16(pb0 + t0, lb);
            dma16(pb1 + t0, lb + 16 * (kGS2 * 2));
        }
    };
    constexpr int MU = DIAG ? 4 : 8, MV = 4;
    int ra = 0, cb = 0;
    if (DIAG) {
        ra = w == 0 ? 0 : w <= 2 ? 1 : w <= 5 ? 2 : 3;
        cb = w == 0 ? 0 : w <= 2 ? w - 1 : w <= 5 ? w - 3 : w - 6;
    }
    const int wr = DIAG ? 64 * ra : 128 * (w >> 2), wc = DIAG ? 64 * cb : 64 * (w & 3);
    float4v acc[MU][MV];
#pragma unroll
    for (int u = 0; u < MU; ++u)
#pragma unroll
        for (int v = 0; v < MV; ++v) acc[u][v] = float4v{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int slot) __attribute__((always_inline)) {
        const uint16_t* Ab = Ar[slot];
        const uint16_t* Bb = DIAG ? Ar[slot] : Br[slot];
        half8 av[MU], bv[MV];
#pragma unroll
        for (int u = 0; u < MU; ++u) {
            const int row = wr + 16 * u + r16;
            av[u] = __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(Ab + row * kGS2 + 8 * gswz(row, q)));
        }
#pragma unroll
        for (int v = 0; v < MV; ++v) {
            const int row = wc + 16 * v + r16;
            bv[v] = __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(Bb + row * kGS2 + 8 * gswz(row, q)));
        }
#pragma unroll
        for (int u = 0; u < MU; ++u)
#pragma unroll
            for (int v = 0; v < MV; ++v)
                acc[u][v] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[u], bv[v], acc[u][v], 0, 0, 0);
    };
    // Stage j sits in ring slot j % 4.  At stage j this wave's loads of stage j
    // are waited for (those of j + 1 and j + 2 stay in flight), the workgroup
    // meets (every wave's loads of j have landed, every wave is done with slot
    // (j - 1) % 4), stage j + 3 is issued into that slot, and j is multiplied.
    const int n = se - sb;
    if (n > 0) issue(sb, 0);
    if (n > 1) issue(sb + 1, 1);
    if (n > 2) issue(sb + 2, 2);
#define GRAM_STEP(j_, slot_)                                                             \
    {                                                                                   \
        const int j = (j_);                                                             \
        if (j + 2 < n) wait_vmem<2 * NDMA>();                                           \
        else if (j + 1 < n) wait_vmem<NDMA>();                                          \
        else wait_vmem<0>();                                                            \
        wg_barrier();                                                                   \
        if (j + 3 < n) issue(sb + j + 3, ((slot_) + 3) % kGRing);                       \
        compute(slot_);                                                                 \
    }
    int s = 0;
    for (; s + kGRing <= n; s += kGRing) {
        GRAM_STEP(s, 0);
        GRAM_STEP(s + 1, 1);
        GRAM_STEP(s + 2, 2);
        GRAM_STEP(s + 3, 3);
    }
    if (s < n) GRAM_STEP(s, 0);
    if (s + 1 < n) GRAM_STEP(s + 1, 1);
    if (s + 2 < n) GRAM_STEP(s + 2, 2);
#undef GRAM_STEP
#pragma unroll
    for (int u = 0; u < MU; ++u)
#pragma unroll
        for (int v = 0; v < MV; ++v)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = arow0 + wr + 16 * u + 4 * q + e;
                const int j = (DIAG ? arow0 : brow0) + wc + 16 * v + r16;
                if (i < K && j < K) {
                    if (DIAG) H[(int64_t)i * K + j] = acc[u][v][e];
                    else unsafeAtomicAdd(H + (int64_t)i * K + j, acc[u][v][e]);
                }
            }
}

__global__ __launch_bounds__(512) void k_gram_regions(const uint16_t* __restrict__ x, int K, int T,
                                                      float* __restrict__ H, int n_items) {
    __shared__ __attribute__((aligned(16))) uint16_t A0[kGS * kGS2], A1[kGS * kGS2], A2[kGS * kGS2], A3[kGS * kGS2];
    __shared__ __attribute__((aligned(16))) uint16_t B0[kGS * kGS2], B1[kGS * kGS2], B2[kGS * kGS2], B3[kGS * kGS2];
    uint16_t* const Ar[kGRing] = {A0, A1, A2, A3};
    uint16_t* const Br[kGRing] = {B0, B1, B2, B3};
    // workgroups are dealt round-robin over the 8 XCDs: give each XCD a
    // contiguous run of items (neighbouring super-rows share panels in its L2)
    const int b = blockIdx.x, qn = n_items / 8, rn = n_items % 8, xcd = b % 8;
    const int item = xcd * qn + min(xcd, rn) + b / 8;
    int np = 1;
    while (np * np < n_items) ++np;
    int a, bsr, half;
    bool diag;
    gram_region_of(item, np, a, bsr, half, diag);
    if (diag) gram_region<true>(x, K, T, H, a, 0, 0, Ar, Br);
    else gram_region<false>(x, K, T, H, a, bsr, half, Ar, Br);
}

// Scratch slot m: 64 x 64 floats in quadrant (m % 4) of the (m / 4)-th strictly
// upper 128 x 128 tile of H (row-major order of tiles); the large-shape path
// writes nothing there before the final mirror.
__device__ inline float* gram_slot(float* H, int K, int m) {
    const int nt = K / 128;
    int u = m >> 2, ti = 0;
    while (u >= nt - 1 - ti) {
        u -= nt - 1 - ti;
        ++ti;
    }
    const int tj = ti + 1 + u;
    return H + (int64_t)(128 * ti + 64 * ((m & 3) >> 1)) * K + 128 * tj + 64 * (m & 1);
}

// Quadrants (3,2) and (3,3) of diagonal region a (rows 192..255 of the region
// against its rows 128..255) over piece p of the calibration columns; four
// waves of 16 rows x 128 columns; partials to slots 2 (a P + p) and + 1.
__global__ __launch_bounds__(256) void k_gram_rest(const uint16_t* __restrict__ x, int K, int T,
                                                   float* __restrict__ H, int P) {
    __shared__ __attribute__((aligned(16))) uint16_t A0[64 * kGS2], A1[64 * kGS2], A2[64 * kGS2], A3[64 * kGS2];
    __shared__ __attribute__((aligned(16))) uint16_t B0[128 * kGS2], B1[128 * kGS2], B2[128 * kGS2], B3[128 * kGS2];
    uint16_t* const Ar[kGRing] = {A0, A1, A2, A3};
    uint16_t* const Br[kGRing] = {B0, B1, B2, B3};
    const int a = blockIdx.x / P, p = blockIdx.x % P;
    const int arow0 = kGS * a + 192, brow0 = kGS * a + 128;
    const int S = T / kGS2;
    const int sb = (int)((int64_t)S * p / P), se = (int)((int64_t)S * (p + 1) / P);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, r16 = lane & 15, q = lane >> 4;
    const int wu = __builtin_amdgcn_readfirstlane(w);
    const int chunk = gswz(lane >> 2, lane & 3);
    const uint16_t* pa = x + (int64_t)min(arow0 + 16 * w + (lane >> 2), K - 1) * T + 8 * chunk;
    const uint16_t* pb0 = x + (int64_t)min(brow0 + 32 * w + (lane >> 2), K - 1) * T + 8 * chunk;
    const uint16_t* pb1 = x + (int64_t)min(brow0 + 32 * w + 16 + (lane >> 2), K - 1) * T + 8 * chunk;
    auto issue = [&](int st, int slot) __attribute__((always_inline)) {
        const int t0 = st * kGS2;
        dma16(pa + t0, lds_address(Ar[slot]) + (uint32_t)(16 * wu) * (kGS2 * 2));
        dma16(pb0 + t0, lds_address(Br[slot]) + (uint32_t)(32 * wu) * (kGS2 * 2));
        dma16(pb1 + t0, lds_address(Br[slot]) + (uint32_t)(32 * wu + 16) * (kGS2 * 2));
    };
    float4v acc[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) acc[v] = float4v{0.f, 0.f, 0.f, 0.f};
    auto compute = [&](int slot) __attribute__((always_inline)) {
        const int ra = 16 * w + r16;
        const half8 av =
            __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(Ar[slot] + ra * kGS2 + 8 * gswz(ra, q)));
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            const int rb = 16 * v + r16;
            const half8 bv =
                __builtin_bit_cast(half8, *reinterpret_cast<const u32x4*>(Br[slot] + rb * kGS2 + 8 * gswz(rb, q)));
            acc[v] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc[v], 0, 0, 0);
        }
    };
    constexpr int NDMA = 3;
    const int n = se - sb;
    if (n > 0) issue(sb, 0);
    if (n > 1) issue(sb + 1, 1);
    if (n > 2) issue(sb + 2, 2);
#define GRAM_STEP(j_, slot_)                                                             \
    {                                                                                   \
        const int j = (j_);                                                             \
        if (j + 2 < n) wait_vmem<2 * NDMA>();                                           \
        else if (j + 1 < n) wait_vmem<NDMA>();                                          \
        else wait_vmem<0>();                                                            \
        wg_barrier();                                                                   \
        if (j + 3 < n) issue(sb + j + 3, ((slot_) + 3) % kGRing);                       \
        compute(slot_);                                                                 \
    }
    int s = 0;
    for (; s + kGRing <= n; s += kGRing) {
        GRAM_STEP(s, 0);
        GRAM_STEP(s + 1, 1);
        GRAM_STEP(s + 2, 2);
        GRAM_STEP(s + 3, 3);
    }
    if (s < n) GRAM_STEP(s, 0);
    if (s + 1 < n) GRAM_STEP(s + 1, 1);
    if (s + 2 < n) GRAM_STEP(s + 2, 2);
#undef GRAM_STEP
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        float* dst = gram_slot(H, K, 2 * (a * P + p) + k);
#pragma unroll
        for (int v = 0; v < 4; ++v)
#pragma unroll
            for (int e = 0; e < 4; ++e) dst[(int64_t)(16 * w + 4 * q + e) * K + 16 * v + r16] = acc[4 * k + v][e];
    }
}

// The pieces of each leftover quadrant summed in piece order into H; workgroup =
// (quadrant L, 16 of its rows).
__global__ __launch_bounds__(256) void k_gram_reduce(float* __restrict__ H, int K, int P) {
    __shared__ float* src[kGPieces];
    const int L = blockIdx.x >> 2, part = blockIdx.x & 3;
    const int a = L >> 1, qd = L & 1;
    if ((int)threadIdx.x < P) src[threadIdx.x] = gram_slot(H, K, 2 * (a * P + (int)threadIdx.x) + qd);
    __syncthreads();
    const int i0 = kGS * a + 192, j0 = kGS * a + 128 + 64 * qd;
    for (int e = threadIdx.x; e < 16 * 64; e += 256) {
        const int r = 16 * part + (e >> 6), c = e & 63;
        float sum = 0.f;
        for (int p = 0; p < P; ++p) sum += src[p][(int64_t)r * K + c];
        if (i0 + r < K && j0 + c < K) H[(int64_t)(i0 + r) * K + j0 + c] = sum;
    }
}

// H[i][j] = H[j][i] for i < j, one lower 64 x 64 tile (or diagonal tile) per workgroup.
__global__ __launch_bounds__(256) void k_gram_mirror(float* __restrict__ H, int K) {
    __shared__ float t[64][65];
    int ti, tj;
    lower_tile((int)blockIdx.x, ti, tj);
    const int i0 = 64 * ti, j0 = 64 * tj;
    const int c = threadIdx.x & 63, r0 = threadIdx.x >> 6;
    float v[16];   // all of a thread's loads in flight before the first LDS write
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = H[(int64_t)(i0 + r0 + 4 * k) * K + j0 + c];
#pragma unroll
    for (int k = 0; k < 16; ++k) t[r0 + 4 * k][c] = v[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int r = r0 + 4 * k, di = j0 + r, dj = i0 + c;
        if (di < dj) H[(int64_t)di * K + dj] = t[c][r];
    }
}

__global__ __launch_bounds__(256) void k_fill_zero(float* __restrict__ p, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = 0.f;
}

// The large-shape path pays five launches and one pass over H; it wins from
// about 1024 channels and 16384 tokens (measured on the shapes in the tests).
bool gram_large(int K, int T) { return K >= 1024 && T >= 16384; }

int gram_large_launch(const uint16_t* x, int K, int T, float* H, hipStream_t s) {
    const int np = (K + kGS - 1) / kGS;
    const int n_items = np * np;
    const int64_t kk = (int64_t)K * K;
    const int zgrid = (int)((kk + 255) / 256 < 4096 ? (kk + 255) / 256 : 4096);
    hipLaunchKernelGGL(k_fill_zero, dim3(zgrid), dim3(256), 0, s, H, kk);
    hipLaunchKernelGGL(k_gram_regions, dim3(n_items), dim3(512), 0, s, x, K, T, H, n_items);
    int n_diag = 0;   // diagonal regions whose quadrant row 3 holds channels
    for (int a = 0; a < np; ++a)
        if (kGS * a + 192 < K) ++n_diag;
    if (n_diag) {
        const int nt = K / 128;
        const int slots = 2 * nt * (nt - 1);   // four per strictly upper 128 x 128 tile
        int P = kGPieces;
        if (P > slots / (2 * n_diag)) P = slots / (2 * n_diag);
        if (P > T / kGS2) P = T / kGS2;
        if (P < 1) return SA_ERR_SHAPE;
        hipLaunchKernelGGL(k_gram_rest, dim3(n_diag * P), dim3(256), 0, s, x, K, T, H, P);
        hipLaunchKernelGGL(k_gram_reduce, dim3(2 * n_diag * 4), dim3(256), 0, s, H, K, P);
    }
    const int n64 = K / 64;
    hipLaunchKernelGGL(k_gram_mirror, dim3(n64 * (n64 + 1) / 2), dim3(256), 0, s, H, K);
    return SA_OK;
}

// ---------------------------------------------------------------- damping, reversal

// lambda = damp * mean(diag(H)) (fp64, one workgroup, fixed order).
__global__ __launch_bounds__(256) void k_damping(const float* __restrict__ H, int K, double damp,
                                                 double* __restrict__ lambda) {
    __shared__ double part[256];
    double s = 0.0;
    for (int k = threadIdx.x; k < K; k += 256) s += (double)H[(int64_t)k * K + k];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int w = 128; w >= 1; w >>= 1) {
        if ((int)threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *lambda = damp * (part[0] / K);
}

// A = J H J + lambda I in fp64 (lower triangle and diagonal), J the reversal:
// A[i][j] = H[K-1-j][K-1-i] for j <= i, from H's lower triangle.  One 64 x 64
// tile of A on or below the diagonal per workgroup, passed through LDS so that
// the reads of H and the writes of A both run along rows.
__global__ __launch_bounds__(256) void k_reverse(const float* __restrict__ H, int K,
                                                 const double* __restrict__ lambda,
                                                 double* __restrict__ A) {
    __shared__ float S[64 * 65];
    int ti, tj;
    lower_tile((int)blockIdx.x, ti, tj);
    const int i0 = 64 * ti, j0 = 64 * tj;
    // source block: rows K - j0 - 64 .. K - j0 - 1, columns K - i0 - 64 .. K - i0 - 1 of H
    const int a0 = K - j0 - 64, c0 = K - i0 - 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int a = a0 + ty + 4 * k, c = c0 + tx;
        v[k] = (a >= 0 && c >= 0 && c <= a) ? H[(int64_t)a * K + c] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) S[(ty + 4 * k) * 65 + tx] = v[k];
    __syncthreads();
    const double lam = *lambda;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int r = ty + 4 * k, i = i0 + r, j = j0 + tx;
        if (i < K && j <= i) {
            double val = (double)S[(63 - tx) * 65 + (63 - r)];
            if (i == j) val += lam;
            A[(int64_t)i * K + j] = val;
        }
    }
}

// ---------------------------------------------------------------- blocked Cholesky (fp64, lower)

constexpr int kNB = 64;             // panel width
constexpr int kNBP = kNB + 1;       // LDS row stride (doubles)

typedef double double4v __attribute__((ext_vector_type(4)));

// Broadcast of lane C's value of v (two readlanes).
template <int C>
__device__ inline double lane_value(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)u, C);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), C);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Broadcast of lane Q's value of v to the four lanes of each quad (DPP quad_perm).
template <int Q>
__device__ inline double quad_value(double v) {
    constexpr int ctrl = Q | (Q << 2) | (Q << 4) | (Q << 6);
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_mov_dpp((int)(uint32_t)u, ctrl, 0xf, 0xf, false);
    const uint32_t hi = __builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), ctrl, 0xf, 0xf, false);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int B, int E, typename F>
__device__ inline void cfor(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        cfor<B + 1, E>(f);
    }
}

// Lanes of one wave exchanging data through LDS: the wave's LDS accesses
// complete in program order, so the exchange needs no hardware barrier, only
// wavefront-scope ordering.  Without it the compiler may move a lane's read of
// another lane's entry across the write that fills it (per thread it can prove
// the two addresses differ).
__device__ inline void lds_exchange() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// 1 / sqrt(p): the hardware estimate (v_rsq_f64) refined by two Newton-Raphson
// steps y <- y + y (1 - p y^2) / 2; p <= 0 gives NaN.  Measured on gfx950 over
// 4 M values against the exact root: the estimate alone within 5.2e-8 relative,
// one step 4.2e-15, two steps 1.4e-16 (under one ulp).
__device__ inline double rsqrt_nr(double p) {
    double y = __builtin_amdgcn_rsq(p);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const double e = fma(-p * y, y, 1.0);
        y = fma(0.5 * y, e, y);
    }
    return y;
}

// Diagonal block [j, j + 64) factored in place by a workgroup of four waves
// (256 threads), blocked: the block sits in LDS (`S`, 64 x 65 doubles, lower
// triangle; rows and columns past the matrix as identity), and for each
// 16-column sub-panel
//  - the first wave factors it right-looking, lane r holding row r's 16
//    entries: at step c, with pivot p (lane c's entry) and rd = 1 / sqrt(p),
//    L[c][c] = p rd, the other lanes scale their entry of column c by rd,
//    publish it in LDS (`col`, 64 doubles) and subtract their multiple of it
//    from their later entries of the sub-panel, reading the column back as
//    broadcasts (at most 15 per step); the next pivot is formed on the side
//    from its own lane's entries, so the LDS round trip stays off the chain
//    of pivots;
//  - the four waves subtract its product with itself from the later columns,
//    16 x 16 blocks of the lower triangle on the fp64 matrix cores.
// Entries above the diagonal are never read.  Every global access is a whole
// row: the lower triangle is stored in place and its transpose in the block's
// upper triangle (row c there = column c of L), which the panel solve reads
// contiguously.  A non-positive pivot gives NaN, which then runs through every
// later value.
__device__ __attribute__((always_inline)) inline void chol_block(double* __restrict__ A, int K, int j,
                                                               double* __restrict__ S, double* __restrict__ col) {
    const int t = threadIdx.x, w = t >> 6, r = t & 63;
    const int nb = min(kNB, K - j);
    {
        const int cl = min(r, nb - 1);
        double v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = A[(int64_t)(j + min(w + 4 * i, nb - 1)) * K + j + cl];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int rr = w + 4 * i;
            S[rr * kNBP + r] = (rr < nb && r < nb && r <= rr) ? v[i] : (rr == r ? 1.0 : 0.0);
        }
    }
    __syncthreads();
    const int li = r & 15, lk = r >> 4;
    cfor<0, 4>([&](auto s_) {
        constexpr int s = decltype(s_)::value;
        constexpr int c0 = 16 * s;
        if (w == 0) {
            double a[16];
            cfor<0, 16>([&](auto k_) {
                constexpr int k = decltype(k_)::value;
                a[k] = S[r * kNBP + c0 + k];
            });
            double p = lane_value<c0>(a[0]);
            cfor<0, 16>([&](auto cc_) {
                constexpr int cc = decltype(cc_)::value;
                constexpr int c = c0 + cc;
                const double rd = rsqrt_nr(p);
                const double l = a[cc] * rd;
                a[cc] = r == c ? p * rd : l;
                col[r] = l;
                lds_exchange();
                if constexpr (cc + 1 < 16) p = lane_value<c + 1>(fma(-l, l, a[cc + 1]));
                constexpr int n = 15 - cc;
                if constexpr (n > 0) {
                    double v[n];
                    cfor<0, n>([&](auto i_) {
                        constexpr int i = decltype(i_)::value;
                        v[i] = col[c + 1 + i];
                    });
                    __builtin_amdgcn_sched_barrier(0);
                    cfor<0, n>([&](auto i_) {
                        constexpr int i = decltype(i_)::value;
                        a[cc + 1 + i] = fma(-l, v[i], a[cc + 1 + i]);
                    });
                }
            });
            cfor<0, 16>([&](auto k_) {
                constexpr int k = decltype(k_)::value;
                S[r * kNBP + c0 + k] = a[k];
            });
        }
        __syncthreads();
        if constexpr (s < 3) {
            // blocks (bi, bj), s < bj <= bi <= 3, numbered row by row over that triangle
            constexpr int m = 3 - s, nblk = m * (m + 1) / 2;
            for (int bk = w; bk < nblk; bk += 4) {
                int bi = 0;
                while ((bi + 1) * (bi + 2) / 2 <= bk) ++bi;
                const int bj = bk - bi * (bi + 1) / 2;
                const int R0 = 16 * (s + 1 + bi), C0 = 16 * (s + 1 + bj);
                double4v acc = (double4v){0.0, 0.0, 0.0, 0.0};
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    const double av = S[(R0 + li) * kNBP + c0 + 4 * kk + lk];
                    const double bv = S[(C0 + li) * kNBP + c0 + 4 * kk + lk];
                    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc, 0, 0, 0);
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) S[(R0 + lk + 4 * q) * kNBP + C0 + li] -= acc[q];
            }
            __syncthreads();
        }
    });
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int rr = w + 4 * i;
        const double v = r <= rr ? S[rr * kNBP + r] : S[r * kNBP + rr];
        if (rr < nb && r < nb) A[(int64_t)(j + rr) * K + j + r] = v;
    }
}

// The first diagonal block; later ones are factored by the trailing update
// that finishes them (k_chol_syrk).
__global__ __launch_bounds__(256) void k_chol_diag(double* __restrict__ A, int K, int j) {
    __shared__ double S[kNB * kNBP];
    __shared__ double col[kNB];
    chol_block(A, K, j, S, col);
}

constexpr int kQS = 18;   // LDS stride (doubles) of one (c, q) run of 16 entries of L11

// Panel below the diagonal block: rows r >= j + 64 solve x L11^T = a, 64 rows
// per workgroup of four waves.  Each row is split over the four lanes of a
// quad: lane l of wave w takes row 16 w + l / 4 and its columns 4 m + (l mod 4),
// m = 0 .. 15, in registers.  Right-looking: at step c the lane holding x_c
// scales it by 1 / L11[c][c], the quad shares it (DPP), and each lane subtracts
// its multiple of column c of L11 from its own later entries.  Column c of L11
// is row c of the block's upper triangle (written there by chol_block), held in
// LDS per quad lane; its entries do not depend on x, so the next step's are read
// during the current step's FMAs.  Launched only where the panel has rows below,
// so the diagonal block is whole.
__global__ __launch_bounds__(256) void k_chol_trsm(double* __restrict__ A, int K, int j) {
    __shared__ double lt[kNB * 4 * kQS];   // lt[(c * 4 + q) * kQS + m] = L11[4 m + q][c] if 4 m + q > c, else 0
    __shared__ double rv[kNB];             // 1 / L11[k][k]
    const int t = threadIdx.x;
    {
        double v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int e = t + 256 * i, c = e >> 6, k = e & 63;
            v[i] = A[(int64_t)(j + c) * K + j + k];
        }
        const double dg = A[(int64_t)(j + (t & 63)) * K + j + (t & 63)];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int e = t + 256 * i, c = e >> 6, k = e & 63;
            lt[(c * 4 + (k & 3)) * kQS + (k >> 2)] = k > c ? v[i] : 0.0;
        }
        if (t < kNB) rv[t] = 1.0 / dg;
    }
    const int w = t >> 6, l = t & 63, q = l & 3;
    const int row = j + kNB + blockIdx.x * kNB + 16 * w + (l >> 2);
    const int rowc = min(row, K - 1);
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) x[m] = A[(int64_t)rowc * K + j + 4 * m + q];
    __syncthreads();
    double rq[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) rq[m] = rv[4 * m + q];
    const double* ltq = lt + q * kQS;
    double cur[16], nxt[16];
    cfor<0, 16>([&](auto m_) {
        constexpr int m = decltype(m_)::value;
        cur[m] = ltq[m];
    });
    cfor<0, kNB>([&](auto c_) {
        constexpr int c = decltype(c_)::value;
        constexpr int m0 = c / 4, q0 = c % 4;
        if constexpr (c + 1 < kNB) {
            cfor<(c + 1) / 4, 16>([&](auto m_) {
                constexpr int m = decltype(m_)::value;
                nxt[m] = ltq[(c + 1) * 4 * kQS + m];
            });
        }
        __builtin_amdgcn_sched_barrier(0);
        const double xc = quad_value<q0>(x[m0] * rq[m0]);
        cfor<m0, 16>([&](auto m_) {
            constexpr int m = decltype(m_)::value;
            x[m] = fma(-xc, cur[m], x[m]);
        });
        x[m0] = q == q0 ? xc : x[m0];
        if constexpr (c + 1 < kNB) {
            cfor<(c + 1) / 4, 16>([&](auto m_) {
                constexpr int m = decltype(m_)::value;
                cur[m] = nxt[m];
            });
        }
    });
    if (row < K) {
#pragma unroll
        for (int m = 0; m < 16; ++m) A[(int64_t)row * K + j + 4 * m + q] = x[m];
    }
}

// Trailing update of the lower triangle: A[r][s] -= sum_c L[r][c] L[s][c] over
// the panel's 64 columns, for 64 x 64 tiles (tr >= ts) below the panel, on the
// fp64 matrix cores.  Each wave takes a 32 x 32 quarter of the tile (2 x 2
// blocks of 16 x 16; a diagonal tile's upper quarter is skipped).  The panel
// rows and the tile's current values are loaded together, every load in flight
// before the first LDS write.  Operand layout of v_mfma_f64_16x16x4_f64: lane l
// holds A[l mod 16][l / 16] and B[l / 16][l mod 16]; result register q holds
// row 4 q + l / 16 of column l mod 16.
__global__ __launch_bounds__(256) void k_chol_syrk(double* __restrict__ A, int K, int j) {
    __shared__ double lr_[kNB * kNBP];
    __shared__ double ls_[kNB * kNBP];
    const int b = blockIdx.x;
    int tr, ts;
    lower_tile(b, tr, ts);
    const int base = j + kNB;
    const int r0 = base + tr * kNB, s0 = base + ts * kNB;
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    const int qr = (w >> 1) * 32, qs = (w & 1) * 32;
    const int li = l & 15, lk = l >> 4;
    const bool live = !(tr == ts && qs > qr);
    double cur[2][2][4];
    {
        // rows past the matrix repeat its last row: their products are never stored
        double vr[16], vs[16];
        const int c = threadIdx.x & 63, rr = threadIdx.x >> 6;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            vr[i] = A[(int64_t)min(r0 + rr + 4 * i, K - 1) * K + j + c];
            vs[i] = A[(int64_t)min(s0 + rr + 4 * i, K - 1) * K + j + c];
        }
        if (live) {
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int v = 0; v < 2; ++v)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int r = min(r0 + qr + 16 * u + lk + 4 * q, K - 1);
                        const int s = min(s0 + qs + 16 * v + li, K - 1);
                        cur[u][v][q] = A[(int64_t)r * K + s];
                    }
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            lr_[(rr + 4 * i) * kNBP + c] = vr[i];
            ls_[(rr + 4 * i) * kNBP + c] = vs[i];
        }
    }
    __syncthreads();
    if (live) {
        double4v acc[2][2];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int v = 0; v < 2; ++v) acc[u][v] = (double4v){0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int c = 0; c < kNB; c += 4) {
            double av[2], bv[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                av[u] = lr_[(qr + 16 * u + li) * kNBP + c + lk];
                bv[u] = ls_[(qs + 16 * u + li) * kNBP + c + lk];
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int v = 0; v < 2; ++v)
                    acc[u][v] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[u], bv[v], acc[u][v], 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int v = 0; v < 2; ++v)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int r = r0 + qr + 16 * u + lk + 4 * q, s = s0 + qs + 16 * v + li;
                    if (r < K && s < K && s <= r) A[(int64_t)r * K + s] = cur[u][v][q] - acc[u][v][q];
                }
    }
    // Tile (0, 0) is the next panel's diagonal block, final once this tile is
    // written: its workgroup factors it while the other tiles are still being
    // updated (one launch per panel fewer, and the factorization off the
    // critical path wherever the update takes longer than it).
    if (b == 0) {
        __syncthreads();
        chol_block(A, K, base, lr_, ls_);
    }
}

// d[k] = 1 / L[K-1-k][K-1-k]: the diagonal of the Cholesky factor of H^-1.
__global__ __launch_bounds__(256) void k_inverse_diag(const double* __restrict__ A, int K,
                                                      double* __restrict__ d) {
    const int k = blockIdx.x * 256 + threadIdx.x;
    if (k < K) d[k] = 1.0 / A[(int64_t)(K - 1 - k) * K + (K - 1 - k)];
}

// ---------------------------------------------------------------- criterion

constexpr int kStatBlocks = 1024;

// Per-block fp64 sums of IS and IS^2 over rows blockIdx.x, blockIdx.x +
// gridDim.x, ...: each thread takes columns t, t + 256, ... of a row, eight
// loads in flight, and adds in a fixed order.
__global__ __launch_bounds__(256) void k_is_partials(const float* __restrict__ w, int N, int K,
                                                     const double* __restrict__ d,
                                                     double* __restrict__ part) {
    __shared__ double s1[256], s2[256];
    double a = 0.0, b = 0.0;
    const int t = threadIdx.x;
    for (int n = blockIdx.x; n < N; n += gridDim.x) {
        const float* wr = w + (int64_t)n * K;
        int k = t;
        for (; k + 7 * 256 < K; k += 8 * 256) {
            float v[8];
            double dv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                v[u] = wr[k + 256 * u];
                dv[u] = d[k + 256 * u];
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const double x = (double)v[u] / dv[u];
                a += x;
                b += x * x;
            }
        }
        for (; k < K; k += 256) {
            const double x = (double)wr[k] / d[k];
            a += x;
            b += x * x;
        }
    }
    s1[t] = a;
    s2[t] = b;
    __syncthreads();
    for (int m = 128; m >= 1; m >>= 1) {
        if (t < m) {
            s1[t] += s1[t + m];
            s2[t] += s2[t + m];
        }
        __syncthreads();
    }
    if (t == 0) {
        part[2 * blockIdx.x] = s1[0];
        part[2 * blockIdx.x + 1] = s2[0];
    }
}

// out[0] = C = ||IS||_F STD(IS)^2, out[1] = ||IS||_F, out[2] = STD(IS).
__global__ __launch_bounds__(256) void k_is_final(const double* __restrict__ part, int nparts,
                                                  int64_t n, double* __restrict__ out) {
    __shared__ double s1[256], s2[256];
    double a = 0.0, b = 0.0;
    for (int p = threadIdx.x; p < nparts; p += 256) {
        a += part[2 * p];
        b += part[2 * p + 1];
    }
    s1[threadIdx.x] = a;
    s2[threadIdx.x] = b;
    __syncthreads();
    for (int m = 128; m >= 1; m >>= 1) {
        if ((int)threadIdx.x < m) {
            s1[threadIdx.x] += s1[threadIdx.x + m];
            s2[threadIdx.x] += s2[threadIdx.x + m];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double mean = s1[0] / (double)n;
        const double var = fmax(s2[0] / (double)n - mean * mean, 0.0);
        const double fro = sqrt(s2[0]);
        out[0] = fro * var;
        out[1] = fro;
        out[2] = sqrt(var);
    }
}

int status() { return hipGetLastError() == hipSuccess ? SA_OK : SA_ERR_HIP; }

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

// ---------------------------------------------------------------- C ABI

SA_API int sa_gram_f16(const uint16_t* x, int K, int T, float* H, void* stream) {
    if (!x || !H) return SA_ERR_NULL;
    if (K < kGT || (K % kGT) || T < kGK || (T % kGK) || (int64_t)K * T > ((int64_t)1 << 40))
        return SA_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(x) & 15u) || (reinterpret_cast<uintptr_t>(H) & 3u))
        return SA_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (gram_large(K, T)) {
        const int rc = gram_large_launch(x, K, T, H, s);
        if (rc != SA_OK) return rc;
        return status();
    }
    const int tiles = K / kGT;
    hipLaunchKernelGGL(k_gram_f16, dim3(tiles * (tiles + 1) / 2), dim3(256), 0, s, x, K, T, H);
    return status();
}

SA_API size_t sa_inverse_cholesky_workspace(int K) {
    if (K < 1) return 0;
    return align256((size_t)K * K * sizeof(double)) + 256;
}

SA_API int sa_inverse_cholesky_diag(const float* H, int K, double damp, double* d,
                                    void* workspace, size_t workspace_bytes, void* stream) {
    if (!H || !d || !workspace) return SA_ERR_NULL;
    if (K < 1 || K > 65536 || !(damp >= 0.0)) return SA_ERR_SHAPE;
    if (workspace_bytes < sa_inverse_cholesky_workspace(K)) return SA_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) || (reinterpret_cast<uintptr_t>(d) & 7u))
        return SA_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    double* A = static_cast<double*>(workspace);
    double* lambda = reinterpret_cast<double*>(static_cast<char*>(workspace) +
                                               align256((size_t)K * K * sizeof(double)));
    hipLaunchKernelGGL(k_damping, dim3(1), dim3(256), 0, s, H, K, damp, lambda);
    const int nt = (K + 63) / 64;
    hipLaunchKernelGGL(k_reverse, dim3(nt * (nt + 1) / 2), dim3(256), 0, s, H, K, lambda, A);
    hipLaunchKernelGGL(k_chol_diag, dim3(1), dim3(256), 0, s, A, K, 0);
    for (int j = 0; j < K; j += kNB) {
        const int below = K - j - kNB;
        if (below > 0) {
            const int rb = (below + kNB - 1) / kNB;
            hipLaunchKernelGGL(k_chol_trsm, dim3((below + 63) / 64), dim3(256), 0, s, A, K, j);
            hipLaunchKernelGGL(k_chol_syrk, dim3(rb * (rb + 1) / 2), dim3(256), 0, s, A, K, j);
        }
    }
    hipLaunchKernelGGL(k_inverse_diag, dim3((K + 255) / 256), dim3(256), 0, s, A, K, d);
    return status();
}

SA_API size_t sa_importance_workspace(void) { return (size_t)2 * kStatBlocks * sizeof(double); }

// The partial sums of sa_importance_criterion_noalloc: a fixed device array
// (16 KB, one per GPU the library runs on, held until the process ends).  In
// host code its name is only a stand-in for the symbol; the device address
// comes from hipGetSymbolAddress, once per device, and only that address is
// handed to kernels.
static __device__ __align__(256) double scratch[2 * kStatBlocks];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
double* g_scratch_ptr[kMaxDevices] = {};

// Address of this device's `scratch` (the current device), or nullptr with
// *status set when the runtime cannot provide it.
double* scratch_on_current_device(int* status) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *status = SA_ERR_HIP;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            *status = SA_ERR_HIP;
            return nullptr;
        }
        g_scratch_ptr[dev] = static_cast<double*>(p);
    }
    *status = SA_OK;
    return g_scratch_ptr[dev];
}

}  // namespace

SA_API int sa_importance_criterion(const float* w, int N, int K, const double* d, double* out,
                                   void* workspace, size_t workspace_bytes, void* stream) {
    if (!w || !d || !out || !workspace) return SA_ERR_NULL;
    if (N < 1 || K < 1 || (int64_t)N * K > ((int64_t)1 << 40)) return SA_ERR_SHAPE;
    if (workspace_bytes < sa_importance_workspace()) return SA_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 7u) || (reinterpret_cast<uintptr_t>(out) & 7u))
        return SA_ERR_ALIGN;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    double* part = static_cast<double*>(workspace);
    hipLaunchKernelGGL(k_is_partials, dim3(kStatBlocks), dim3(256), 0, s, w, N, K, d, part);
    hipLaunchKernelGGL(k_is_final, dim3(1), dim3(256), 0, s, part, kStatBlocks, (int64_t)N * K,
                       out);
    return status();
}

SA_API int sa_importance_criterion_noalloc(const float* w, int N, int K, const double* d,
                                           double* out, void* stream) {
    if (!w || !d || !out) return SA_ERR_NULL;
    if (N < 1 || K < 1 || (int64_t)N * K > ((int64_t)1 << 40)) return SA_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(out) & 7u) return SA_ERR_ALIGN;
    int st = SA_OK;
    double* part = scratch_on_current_device(&st);
    if (!part) return st;
    // the same kernels as sa_importance_criterion; every partial is written
    // before it is read, so nothing needs clearing between calls
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipLaunchKernelGGL(k_is_partials, dim3(kStatBlocks), dim3(256), 0, s, w, N, K, d, part);
    hipLaunchKernelGGL(k_is_final, dim3(1), dim3(256), 0, s, part, kStatBlocks, (int64_t)N * K,
                       out);
    return status();
}

// ---------------------------------------------------------------- host: fits and Eq. 4

SA_API int sa_fit_per_bit(const double* c, const double* errors, int L, int nb, int degree,
                          double* out) {
    if (!c || !errors || !out) return SA_ERR_NULL;
    if (L < 1 || nb < 1 || degree < 0 || degree > 8 || L < degree + 1) return SA_ERR_SHAPE;
    const int m = degree + 1;
    // least squares by the normal equations of the scaled Vandermonde system
    // (columns c^p / s^p, s = max |c|), solved by Gaussian elimination with
    // partial pivoting in fp64
    double sc = 0.0;
    for (int i = 0; i < L; ++i) sc = fmax(sc, fabs(c[i]));
    if (sc == 0.0) sc = 1.0;
    std::vector<double> M(m * m), v(m), coef(m);
    for (int b = 0; b < nb; ++b) {
        std::fill(M.begin(), M.end(), 0.0);
        std::fill(v.begin(), v.end(), 0.0);
        for (int i = 0; i < L; ++i) {
            const double t = c[i] / sc;
            double pp[9];
            pp[0] = 1.0;
            for (int p = 1; p < m; ++p) pp[p] = pp[p - 1] * t;
            for (int p = 0; p < m; ++p) {
                v[p] += pp[p] * errors[i * nb + b];
                for (int q = 0; q < m; ++q) M[p * m + q] += pp[p] * pp[q];
            }
        }
        for (int col = 0; col < m; ++col) {
            int piv = col;
            for (int r = col + 1; r < m; ++r)
                if (fabs(M[r * m + col]) > fabs(M[piv * m + col])) piv = r;
            if (M[piv * m + col] == 0.0) return SA_ERR_SHAPE;  // too few distinct criteria
            if (piv != col) {
                for (int q = 0; q < m; ++q) std::swap(M[piv * m + q], M[col * m + q]);
                std::swap(v[piv], v[col]);
            }
            for (int r = col + 1; r < m; ++r) {
                const double f = M[r * m + col] / M[col * m + col];
                for (int q = col; q < m; ++q) M[r * m + q] -= f * M[col * m + q];
                v[r] -= f * v[col];
            }
        }
        for (int col = m - 1; col >= 0; --col) {
            double acc = v[col];
            for (int q = col + 1; q < m; ++q) acc -= M[col * m + q] * coef[q];
            coef[col] = acc / M[col * m + col];
        }
        for (int i = 0; i < L; ++i) {
            const double t = c[i] / sc;
            double y = 0.0;
            for (int p = m - 1; p >= 0; --p) y = y * t + coef[p];
            out[i * nb + b] = y;
        }
    }
    return SA_OK;
}

SA_API int sa_allocate_bits(const double* cost, const int* bits, int L, int nb, double budget,
                            int* out, double* objective) {
    if (!cost || !bits || !out) return SA_ERR_NULL;
    if (L < 1 || nb < 1 || nb > 16 || L > 100000) return SA_ERR_SHAPE;
    int bmax = 0;
    for (int k = 0; k < nb; ++k) {
        if (bits[k] < 1 || bits[k] > 64) return SA_ERR_SHAPE;
        bmax = bits[k] > bmax ? bits[k] : bmax;
    }
    // a total t is allowed when t <= budget * L in fp64, i.e. t <= floor(budget * L)
    const double capd = floor(budget * (double)L);
    if (!(capd >= 0.0)) return SA_ERR_SHAPE;
    const int64_t cap = (int64_t)fmin(capd, (double)bmax * L);
    const int64_t W = cap + 1;
    // f[l][t]: the best prefix over layers 0..l-1 using exactly t bits -- the
    // smallest objective (summed from layer 0), then the lexicographically
    // smallest widths; choice[l][t] is the last layer's option of that prefix.
    const double INF = INFINITY;
    std::vector<double> f((size_t)(L + 1) * W, INF);
    std::vector<int8_t> choice((size_t)(L + 1) * W, -1);
    f[0] = 0.0;
    auto lex_less = [&](int l, int64_t t1, int k1, int64_t t2, int k2) {
        // compare the widths of prefix (l, t1 via k1) with (l, t2 via k2), both of l + 1 layers
        std::vector<int> a(l + 1), b(l + 1);
        int64_t u = t1;
        a[l] = bits[k1];
        u -= bits[k1];
        for (int m = l - 1; m >= 0; --m) {
            const int k = choice[(size_t)(m + 1) * W + u];
            a[m] = bits[k];
            u -= bits[k];
        }
        u = t2;
        b[l] = bits[k2];
        u -= bits[k2];
        for (int m = l - 1; m >= 0; --m) {
            const int k = choice[(size_t)(m + 1) * W + u];
            b[m] = bits[k];
            u -= bits[k];
        }
        return a < b;
    };
    for (int l = 0; l < L; ++l) {
        for (int64_t t = 0; t < W; ++t) {
            const double base = f[(size_t)l * W + t];
            if (base == INF) continue;
            for (int k = 0; k < nb; ++k) {
                const int64_t t2 = t + bits[k];
                if (t2 >= W) continue;
                const double v = base + cost[(size_t)l * nb + k];
                double& cur = f[(size_t)(l + 1) * W + t2];
                int8_t& ch = choice[(size_t)(l + 1) * W + t2];
                if (v < cur || (v == cur && ch >= 0 && lex_less(l, t2, k, t2, ch))) {
                    cur = v;
                    ch = (int8_t)k;
                }
            }
        }
    }
    int64_t best_t = -1;
    for (int64_t t = 0; t < W; ++t) {
        const double v = f[(size_t)L * W + t];
        if (v == INF) continue;
        if (best_t < 0 || v < f[(size_t)L * W + best_t]) best_t = t;  // ties: fewer bits
    }
    if (best_t < 0) return SA_ERR_SHAPE;  // nothing fits the budget
    int64_t u = best_t;
    for (int l = L - 1; l >= 0; --l) {
        const int k = choice[(size_t)(l + 1) * W + u];
        out[l] = bits[k];
        u -= bits[k];
    }
    if (objective) *objective = f[(size_t)L * W + best_t];
    return SA_OK;
}
