// gfx950 kernel and C ABI of the offline reparameterization of ShiftAddLLM:
// full-precision weights -> the shift-add layer's sign planes and power-of-two
// exponents.
//
// Alternating multi-bit binary-coding quantization (Sec. 3, Alg. 1) with every
// scale factor a power of two (Sec. 4.1, Eq. 2, one term).  Each segment of G
// consecutive columns of one row of W is quantized on its own, in fp64:
//   greedy (Eq. 1):  r = w; for i < q: b_i = sign(r) (sign(0) = +1),
//                    alpha_i = sum|r| / G, r -= alpha_i b_i;
//   T cycles of:     LS  alpha = (B^T B)^-1 B^T w, Gaussian elimination with
//                        partial pivoting (first largest pivot); a column
//                        whose pivot is at most 1e-9 G depends on the earlier
//                        ones and gets alpha = 0;
//                    PoT alpha -> sign * 2^P, P = E + [m >= sqrt 2] for
//                        |alpha| = m 2^E, m in [1, 2) (0 -> P = -128);
//                    BS  each element takes the code whose value
//                        sum_i (+-alpha_i) is nearest (ties: smaller code).
// With T = 0 the greedy scales are rounded to powers of two.  Every step keeps
// the operation order of the definition above, so the only difference between
// runs on different hardware is the order of the two segment sums (sum|r| and
// B^T w).
//
// One wave per segment.  Element k of a segment is always handled by lane
// k mod 64; between passes its code byte (bit i set: b_i = +1) lives in the
// first output plane at the element's own position, read back only by the lane
// that wrote it.  The q x q solve and the table of the 2^q code values are
// wave-uniform and sit in the wave's own LDS region.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "shiftadd.h"

namespace {

constexpr int kQuantThreads = 256;  // 4 waves = 4 segments per workgroup
constexpr int kWaves = kQuantThreads / 64;

__device__ inline double wave_sum_f64(double v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ inline int wave_sum_i32(int v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

// Orders the wave's LDS writes before its later LDS reads of other lanes' data.
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Nearest power of two in the log domain: sign * 2^P, P in [-128, 127].
__device__ inline double pot_value(double a, int* P_out) {
    const double mag = fabs(a);
    if (mag == 0.0) {
        *P_out = -128;
        return 0.0;
    }
    int E;
    const double m = frexp(mag, &E);  // mag = m 2^E, m in [0.5, 1)
    int P = (E - 1) + (2.0 * m >= 1.4142135623730951 ? 1 : 0);
    P = P < -128 ? -128 : (P > 127 ? 127 : P);
    *P_out = P;
    const double v = ldexp(1.0, P);
    return a < 0 ? -v : v;
}

// LS step on the wave's q x q system (every lane runs it on the same values).
template <int Q>
__device__ void solve_ls(double (*a)[Q], double* rhs, double* alpha, double tol) {
    int piv_row[Q], piv_col[Q];
    int kept = 0, row = 0;
    for (int col = 0; col < Q && row < Q; ++col) {
        int p = row;
        double best = fabs(a[row][col]);
        for (int r2 = row + 1; r2 < Q; ++r2) {
            const double v = fabs(a[r2][col]);
            if (v > best) {
                best = v;
                p = r2;
            }
        }
        if (best <= tol) continue;  // dependent column: alpha = 0
        if (p != row) {
            for (int c2 = 0; c2 < Q; ++c2) {
                const double t = a[row][c2];
                a[row][c2] = a[p][c2];
                a[p][c2] = t;
            }
            const double t = rhs[row];
            rhs[row] = rhs[p];
            rhs[p] = t;
        }
        for (int r2 = row + 1; r2 < Q; ++r2) {
            const double f = a[r2][col] / a[row][col];
            for (int c2 = 0; c2 < Q; ++c2) a[r2][c2] = a[r2][c2] - f * a[row][c2];
            rhs[r2] = rhs[r2] - f * rhs[row];
        }
        piv_row[kept] = row;
        piv_col[kept] = col;
        ++kept;
        ++row;
    }
    for (int i = 0; i < Q; ++i) alpha[i] = 0.0;
    for (int t = kept - 1; t >= 0; --t) {
        const int r0 = piv_row[t], c0 = piv_col[t];
        double acc = rhs[r0];
        for (int u = t + 1; u < kept; ++u) acc = acc - a[r0][piv_col[u]] * alpha[piv_col[u]];
        alpha[c0] = acc / a[r0][c0];
    }
}

template <int Q>
__global__ __launch_bounds__(kQuantThreads) void k_quantize_bcq(
    const float* __restrict__ w, int N, int K, int G, int cycles, int8_t* __restrict__ signs,
    int8_t* __restrict__ exps) {
    __shared__ double s_val[kWaves][1 << Q];
    __shared__ double s_a[kWaves][Q][Q];
    __shared__ double s_rhs[kWaves][Q];
    __shared__ double s_alpha[kWaves][Q];

    const int lane = threadIdx.x & 63;
    const int wv = threadIdx.x >> 6;
    const int NG = K / G;
    const int64_t seg = (int64_t)blockIdx.x * kWaves + wv;
    if (seg >= (int64_t)N * NG) return;  // whole wave
    const int n = (int)(seg / NG), g = (int)(seg % NG);
    const float* ws = w + (int64_t)n * K + (int64_t)g * G;
    const int64_t plane = (int64_t)N * K;
    int8_t* cs = signs + (int64_t)n * K + (int64_t)g * G;  // plane i at cs + i * plane
    uint8_t* code = reinterpret_cast<uint8_t*>(cs);        // code bytes, plane 0

    // greedy initialisation (Eq. 1), one pass and one wave sum per plane
    double alpha[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) {
        double part = 0.0;
        for (int k = lane; k < G; k += 64) {
            uint32_t c = i ? code[k] : 0u;
            double r = (double)ws[k];
#pragma unroll
            for (int j = 0; j < i; ++j) r = r - ((c >> j) & 1u ? alpha[j] : -alpha[j]);
            c |= (r >= 0.0 ? 1u : 0u) << i;
            code[k] = (uint8_t)c;
            part += fabs(r);
        }
        alpha[i] = wave_sum_f64(part) / G;
    }
    double pa[Q];
    int P[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) pa[i] = pot_value(alpha[i], &P[i]);

    for (int t = 0; t < cycles; ++t) {
        // LS: B^T w, and B^T B from the disagreements of each pair of planes
        double v[Q];
        int d[Q][Q];
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            v[i] = 0.0;
#pragma unroll
            for (int j = 0; j < Q; ++j) d[i][j] = 0;
        }
        for (int k = lane; k < G; k += 64) {
            const uint32_t c = code[k];
            const double wk = (double)ws[k];
#pragma unroll
            for (int i = 0; i < Q; ++i) {
                v[i] += (c >> i) & 1u ? wk : -wk;
#pragma unroll
                for (int j = i + 1; j < Q; ++j) d[i][j] += (int)(((c >> i) ^ (c >> j)) & 1u);
            }
        }
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const double vi = wave_sum_f64(v[i]);
            if (lane == 0) {
                s_rhs[wv][i] = vi;
                s_a[wv][i][i] = (double)G;
            }
#pragma unroll
            for (int j = i + 1; j < Q; ++j) {
                const double m = (double)(G - 2 * wave_sum_i32(d[i][j]));
                if (lane == 0) s_a[wv][i][j] = s_a[wv][j][i] = m;
            }
        }
        wave_sync();
        if (lane == 0) solve_ls<Q>(s_a[wv], s_rhs[wv], s_alpha[wv], 1e-9 * G);
        wave_sync();
        // PoT, then the table of code values sum_i +-pa_i (in plane order)
#pragma unroll
        for (int i = 0; i < Q; ++i) pa[i] = pot_value(s_alpha[wv][i], &P[i]);
        for (int c = lane; c < (1 << Q); c += 64) {
            double val = 0.0;
#pragma unroll
            for (int i = 0; i < Q; ++i) val = val + ((c >> i) & 1 ? pa[i] : -pa[i]);
            s_val[wv][c] = val;
        }
        wave_sync();
        // BS: nearest code value, first one on ties
        for (int k = lane; k < G; k += 64) {
            const double wk = (double)ws[k];
            double best = fabs(wk - s_val[wv][0]);
            uint32_t bc = 0;
            for (int c = 1; c < (1 << Q); ++c) {
                const double dist = fabs(wk - s_val[wv][c]);
                if (dist < best) {
                    best = dist;
                    bc = (uint32_t)c;
                }
            }
            code[k] = (uint8_t)bc;
        }
        wave_sync();  // the next cycle's table overwrites s_val
    }
    // layer format: planes s_i = sign(pa_i) b_i, exponents P_i
    for (int k = lane; k < G; k += 64) {
        const uint32_t c = code[k];
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const int b = (c >> i) & 1u ? 1 : -1;
            cs[i * plane + k] = (int8_t)(pa[i] < 0 ? -b : b);
        }
    }
    if (lane < Q) {
        int Pi = P[0];
#pragma unroll
        for (int i = 1; i < Q; ++i) Pi = lane == i ? P[i] : Pi;
        exps[((int64_t)lane * N + n) * NG + g] = (int8_t)Pi;
    }
}

template <int Q>
void launch(const float* w, int N, int K, int G, int cycles, int8_t* signs, int8_t* exps,
            unsigned grid, hipStream_t s) {
    hipLaunchKernelGGL(k_quantize_bcq<Q>, dim3(grid), dim3(kQuantThreads), 0, s, w, N, K, G,
                       cycles, signs, exps);
}

}  // namespace

SA_API int sa_quantize_bcq(const float* w, int N, int K, int q, int group, int cycles,
                           int8_t* signs, int8_t* exps, void* stream) {
    if (!w || !signs || !exps) return SA_ERR_NULL;
    if (q < 1 || q > SA_MAX_Q) return SA_ERR_Q;
    if (N < 1 || K < 8 || (K & 7)) return SA_ERR_SHAPE;
    if ((int64_t)q * N * K > (int64_t)1 << 36) return SA_ERR_SHAPE;
    if ((int64_t)N * (K / 8) >= (int64_t)1 << 31) return SA_ERR_SHAPE;
    if (group < 8 || (group & 7) || (K % group)) return SA_ERR_GROUP;
    if (cycles < 0 || cycles > SA_MAX_CYCLES) return SA_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(w) & 3u) return SA_ERR_ALIGN;
    const int64_t segs = (int64_t)N * (K / group);
    const int64_t grid = (segs + kWaves - 1) / kWaves;
    if (grid > 0x7fffffff) return SA_ERR_SHAPE;
    const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const unsigned gd = (unsigned)grid;
    switch (q) {
        case 1: launch<1>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 2: launch<2>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 3: launch<3>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 4: launch<4>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 5: launch<5>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 6: launch<6>(w, N, K, group, cycles, signs, exps, gd, s); break;
        case 7: launch<7>(w, N, K, group, cycles, signs, exps, gd, s); break;
        default: launch<8>(w, N, K, group, cycles, signs, exps, gd, s); break;
    }
    return hipGetLastError() == hipSuccess ? SA_OK : SA_ERR_HIP;
}
