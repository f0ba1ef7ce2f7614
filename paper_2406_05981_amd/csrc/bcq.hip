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
// Two kernels, the same arithmetic:
//  * k_quantize_seg (group <= 256): LN lanes per segment (4, 8 or 16).  Lane l
//    holds E consecutive weights of its segment in registers for the whole run
//    and the codes as one bit mask per plane, so the weights are read once and
//    the planes written once.  Segment sums are reduced across the lanes of a
//    DPP row; B^T B comes from popcounts of mask pairs.
//  * k_quantize_bcq (any group): one wave per segment; element k is handled by
//    lane k mod 64 and its code byte (bit i set: b_i = +1) lives in the first
//    output plane between passes, read back only by the lane that wrote it.
// Every lane of a segment sees the same bits of every sum (each reduction step
// adds a pair of partial sums in both lanes of the pair; addition commutes).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <type_traits>

#include "shiftadd.h"

namespace {

constexpr int kQuantThreads = 256;  // 4 waves = 4 segments per workgroup
constexpr int kWaves = kQuantThreads / 64;
constexpr int kSegMaxGroup = 256;   // largest group of the register kernel
constexpr int kRegSolveMaxQ = 4;     // largest q solved in registers
constexpr int kSegMaxBlocks = 2048;  // workgroups of the register kernel; each group loops

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

// Additive PoT (Eq. 2 with `terms` terms): term t is the PoT of the residual
// the previous terms leave.  Returns the value (summed in term order from 0);
// packs each term's exponent and sign (+-1, 0 for a zero residual) into byte t
// of *pe and *ps.  One term is pot_value.
__device__ inline double pot_terms(double a, int terms, uint32_t* pe, uint32_t* ps) {
    double r = a, val = 0.0;
    uint32_t e = 0, sg = 0;
#pragma unroll
    for (int t = 0; t < SA_MAX_TERMS; ++t) {
        if (t < terms) {
            int P;
            const double v = pot_value(r, &P);
            const int s1 = r == 0.0 ? 0 : (r < 0.0 ? -1 : 1);
            e |= (uint32_t)(uint8_t)(int8_t)P << (8 * t);
            sg |= (uint32_t)(uint8_t)(int8_t)s1 << (8 * t);
            val = val + v;
            r = r - v;
        }
    }
    *pe = e;
    *ps = sg;
    return val;
}

// Writes the exponents (and, when tsg is given, the term signs relative to the
// first term, whose sign goes into the plane) of one segment: plane i, term t
// at offset i * ex_plane * terms + t (the terms of a segment are consecutive).
template <int Q>
__device__ inline void write_scales(const uint32_t (&pe)[Q], const uint32_t (&ps)[Q], int terms,
                                    int8_t* __restrict__ ex, int8_t* __restrict__ tsg,
                                    int64_t ex_plane) {
#pragma unroll
    for (int i = 0; i < Q; ++i) {
        const int s0 = (int8_t)(ps[i] & 0xffu) < 0 ? -1 : 1;
#pragma unroll
        for (int t = 0; t < SA_MAX_TERMS; ++t) {
            if (t < terms) {
                const int64_t at = i * ex_plane * terms + t;
                ex[at] = (int8_t)(pe[i] >> (8 * t));
                if (tsg) tsg[at] = (int8_t)((int)(int8_t)(ps[i] >> (8 * t)) * s0);
            }
        }
    }
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

// Compile-time loop: f(std::integral_constant<int, i>) for i in [B, E).  Array
// indices stay constants from the start, so the arrays of the register solve
// are never given a run-time index (which would move them out of registers).
template <int B, int E, typename F>
__device__ inline void sfor(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        sfor<B + 1, E>(f);
    }
}

// The same LS step in registers, for the common case in which no column is
// dependent (every pivot above tol).  Row swaps are selects over the rows that
// are still candidates; the entries left of the pivot column are never read
// again by the elimination or the back substitution, so they are not updated.
// Returns false when a pivot is at most tol (the caller then runs solve_ls).
template <int Q>
__device__ inline bool solve_ls_regs(double (&a)[Q][Q], double (&rhs)[Q], double (&alpha)[Q],
                                     double tol) {
    bool ok = true;
    sfor<0, Q>([&](auto col_) {
        constexpr int col = decltype(col_)::value;
        uint32_t pm = 1u << col;  // pivot row, one-hot
        double best = fabs(a[col][col]);
        sfor<col + 1, Q>([&](auto r_) {
            constexpr int r = decltype(r_)::value;
            const double v = fabs(a[r][col]);
            pm = v > best ? 1u << r : pm;
            best = v > best ? v : best;
        });
        ok = ok && best > tol;
        sfor<col, Q>([&](auto c_) {
            constexpr int c = decltype(c_)::value;
            double pv = a[col][c];
            sfor<col + 1, Q>([&](auto r_) {
                constexpr int r = decltype(r_)::value;
                pv = (pm >> r) & 1u ? a[r][c] : pv;
                a[r][c] = (pm >> r) & 1u ? a[col][c] : a[r][c];
            });
            a[col][c] = pv;
        });
        {
            double pv = rhs[col];
            sfor<col + 1, Q>([&](auto r_) {
                constexpr int r = decltype(r_)::value;
                pv = (pm >> r) & 1u ? rhs[r] : pv;
                rhs[r] = (pm >> r) & 1u ? rhs[col] : rhs[r];
            });
            rhs[col] = pv;
        }
        sfor<col + 1, Q>([&](auto r_) {
            constexpr int r2 = decltype(r_)::value;
            const double f = a[r2][col] / a[col][col];
            sfor<col + 1, Q>([&](auto c_) {
                constexpr int c = decltype(c_)::value;
                a[r2][c] = a[r2][c] - f * a[col][c];
            });
            rhs[r2] = rhs[r2] - f * rhs[col];
        });
    });
    sfor<0, Q>([&](auto k_) {
        constexpr int col = Q - 1 - decltype(k_)::value;
        double acc = rhs[col];
        sfor<col + 1, Q>([&](auto c_) {
            constexpr int c = decltype(c_)::value;
            acc = acc - a[col][c] * alpha[c];
        });
        alpha[col] = acc / a[col][col];
    });
    return ok;
}

template <int Q>
__global__ __launch_bounds__(kQuantThreads) void k_quantize_bcq(
    const float* __restrict__ w, int N, int K, int G, int cycles, int terms,
    int8_t* __restrict__ signs, int8_t* __restrict__ exps, int8_t* __restrict__ tsg) {
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
    uint32_t pe[Q], ps[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) pa[i] = pot_terms(alpha[i], terms, &pe[i], &ps[i]);

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
        for (int i = 0; i < Q; ++i) pa[i] = pot_terms(s_alpha[wv][i], terms, &pe[i], &ps[i]);
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
    // layer format: planes s_i = (sign of the first term of pa_i) b_i, exponents
    // (and term signs) per term
    for (int k = lane; k < G; k += 64) {
        const uint32_t c = code[k];
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            const int b = (c >> i) & 1u ? 1 : -1;
            cs[i * plane + k] = (int8_t)((int8_t)(ps[i] & 0xffu) < 0 ? -b : b);
        }
    }
    if (lane == 0) {
        const int64_t at = ((int64_t)n * NG + g) * terms;
        write_scales<Q>(pe, ps, terms, exps + at, tsg ? tsg + at : nullptr, (int64_t)N * NG);
    }
}

// ------------------------------------------------ a few lanes per segment

template <int CTRL>
__device__ inline int dpp_i32(int v) {
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, false);
}

template <int CTRL>
__device__ inline double dpp_f64(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)u);
    const uint32_t hi = (uint32_t)dpp_i32<CTRL>((int)(uint32_t)(u >> 32));
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Sum over the LN lanes (4, 8 or 16) of a segment inside one DPP row: swap
// neighbours, swap pairs, then mirror within 8 and within 16 lanes.  Every
// lane of the segment ends with the same bits.
template <int LN>
__device__ inline double seg_sum(double v) {
    v = v + dpp_f64<0xB1>(v);                             // quad_perm(1, 0, 3, 2)
    v = v + dpp_f64<0x4E>(v);                             // quad_perm(2, 3, 0, 1)
    if constexpr (LN >= 8) v = v + dpp_f64<0x141>(v);     // row_half_mirror
    if constexpr (LN >= 16) v = v + dpp_f64<0x140>(v);    // row_mirror
    return v;
}

template <int LN>
__device__ inline int seg_sum_i32(int v) {
    v = v + dpp_i32<0xB1>(v);
    v = v + dpp_i32<0x4E>(v);
    if constexpr (LN >= 8) v = v + dpp_i32<0x141>(v);
    if constexpr (LN >= 16) v = v + dpp_i32<0x140>(v);
    return v;
}

// +x or -x by the sign bit alone (exactly the negation, zeros included)
__device__ inline double with_sign(double x, bool neg) {
    return __builtin_bit_cast(double,
                              __builtin_bit_cast(uint64_t, x) ^ ((uint64_t)(neg ? 1u : 0u) << 63));
}

template <int Q, int LN>
struct SegLds {
    static constexpr int kSegs = kQuantThreads / LN;
    double a[kSegs][Q][Q];
    double rhs[kSegs][Q];
    double alpha[kSegs][Q];
    double val[Q > 4 ? kSegs : 1][Q > 4 ? (1 << Q) : 1];
};

// One segment, weights already in registers: lane l holds the E consecutive
// elements l E .. l E + E - 1 (slot e = element l E + e; 0 in an empty slot).
// FULL: no empty slot (G == LN E).  Otherwise empty slots come in whole runs
// of 8, since G is a multiple of 8 and E is 8 or more.
template <int Q, int E, int LN, bool FULL>
__device__ inline void quantize_segment(const float (&wf)[E], int l, int sb, int G, int cycles,
                                        int terms, int8_t* __restrict__ cs, int64_t plane,
                                        int8_t* __restrict__ ex, int8_t* __restrict__ tsg,
                                        int64_t ex_plane, SegLds<Q, LN>& lds) {
    constexpr int NV = 1 << Q;
    constexpr bool kTableInLds = Q > 4;
    auto& s_a = lds.a;
    auto& s_rhs = lds.rhs;
    auto& s_alpha = lds.alpha;
    auto& s_val = lds.val;
    uint32_t vm = E >= 32 ? ~0u : (1u << E) - 1;  // valid slots
    if constexpr (!FULL) {
        vm = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) vm |= (l * E + e < G ? 1u : 0u) << e;
    }

    // greedy initialisation (Eq. 1); the residual of plane i is rebuilt from w
    // with the same subtractions in the same order
    uint32_t m[Q];
    double alpha[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) {
        uint32_t mi = 0;
        double part = 0.0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            double r = (double)wf[e];
#pragma unroll
            for (int j = 0; j < i; ++j) r = r - with_sign(alpha[j], !((m[j] >> e) & 1u));
            mi |= (r >= 0.0 ? 1u : 0u) << e;
            if (FULL || ((vm >> e) & 1u)) part += fabs(r);
        }
        alpha[i] = seg_sum<LN>(part) / G;
        m[i] = mi & vm;
    }
    double pa[Q];
    uint32_t pe[Q], ps[Q];
#pragma unroll
    for (int i = 0; i < Q; ++i) pa[i] = pot_terms(alpha[i], terms, &pe[i], &ps[i]);

    for (int t = 0; t < cycles; ++t) {
        // LS: B^T w per plane, B^T B from popcounts of mask pairs
        double v[Q];
#pragma unroll
        for (int i = 0; i < Q; ++i) v[i] = 0.0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            // an empty slot holds w = 0 and adds +-0, which leaves the sum as is
            const double wd = (double)wf[e];
#pragma unroll
            for (int i = 0; i < Q; ++i) v[i] += with_sign(wd, !((m[i] >> e) & 1u));
        }
        // disagreement counts of the plane pairs (i < j), three 10-bit fields
        // per word (a count is at most G <= 256)
        constexpr int NP = Q * (Q - 1) / 2, NW = (NP + 2) / 3;
        int pw[NW > 0 ? NW : 1];
#pragma unroll
        for (int u = 0; u < NW; ++u) pw[u] = 0;
        {
            int pi = 0;
#pragma unroll
            for (int i = 0; i < Q; ++i)
#pragma unroll
                for (int j = i + 1; j < Q; ++j, ++pi)
                    pw[pi / 3] += __builtin_popcount(m[i] ^ m[j]) << (10 * (pi % 3));
        }
#pragma unroll
        for (int u = 0; u < NW; ++u) pw[u] = seg_sum_i32<LN>(pw[u]);
        double a[Q][Q], rhs[Q], al[Q];
#pragma unroll
        for (int i = 0; i < Q; ++i) {
            rhs[i] = seg_sum<LN>(v[i]);
            a[i][i] = (double)G;
        }
        {
            int pi = 0;
#pragma unroll
            for (int i = 0; i < Q; ++i)
#pragma unroll
                for (int j = i + 1; j < Q; ++j, ++pi)
                    a[i][j] = a[j][i] = (double)(G - 2 * ((pw[pi / 3] >> (10 * (pi % 3))) & 1023));
        }
        bool ok = false;
        if constexpr (Q <= kRegSolveMaxQ) {
            double a2[Q][Q], r2[Q];
#pragma unroll
            for (int i = 0; i < Q; ++i) {
                r2[i] = rhs[i];
#pragma unroll
                for (int j = 0; j < Q; ++j) a2[i][j] = a[i][j];
            }
            ok = solve_ls_regs<Q>(a2, r2, al, 1e-9 * G);
        }
        if (!ok) {  // a dependent column (or a large q): the general solve in LDS
            if (l == 0) {
#pragma unroll
                for (int i = 0; i < Q; ++i) {
                    s_rhs[sb][i] = rhs[i];
#pragma unroll
                    for (int j = 0; j < Q; ++j) s_a[sb][i][j] = a[i][j];
                }
                solve_ls<Q>(s_a[sb], s_rhs[sb], s_alpha[sb], 1e-9 * G);
            }
            wave_sync();
#pragma unroll
            for (int i = 0; i < Q; ++i) al[i] = s_alpha[sb][i];
        }
#pragma unroll
        for (int i = 0; i < Q; ++i) pa[i] = pot_terms(al[i], terms, &pe[i], &ps[i]);

        // BS against the 2^q code values sum_i +-pa_i (plane order)
        uint32_t mn[Q];
#pragma unroll
        for (int i = 0; i < Q; ++i) mn[i] = 0;
        if constexpr (!kTableInLds) {
            double val[NV];
#pragma unroll
            for (int c = 0; c < NV; ++c) {
                double a = 0.0;
#pragma unroll
                for (int i = 0; i < Q; ++i) a = a + ((c >> i) & 1 ? pa[i] : -pa[i]);
                val[c] = a;
            }
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const double wd = (double)wf[e];
                double best = fabs(wd - val[0]);
                uint32_t bc = 0;
#pragma unroll
                for (int c = 1; c < NV; ++c) {
                    const double d = fabs(wd - val[c]);
                    bc = d < best ? (uint32_t)c : bc;
                    best = fmin(d, best);  // equal only when d == best: same bits
                }
#pragma unroll
                for (int i = 0; i < Q; ++i) mn[i] |= ((bc >> i) & 1u) << e;
            }
        } else {
            for (int c = l; c < NV; c += LN) {
                double a = 0.0;
#pragma unroll
                for (int i = 0; i < Q; ++i) a = a + ((c >> i) & 1 ? pa[i] : -pa[i]);
                s_val[sb][c] = a;
            }
            wave_sync();
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const double wd = (double)wf[e];
                double best = fabs(wd - s_val[sb][0]);
                uint32_t bc = 0;
                for (int c = 1; c < NV; ++c) {
                    const double d = fabs(wd - s_val[sb][c]);
                    bc = d < best ? (uint32_t)c : bc;
                    best = d < best ? d : best;
                }
#pragma unroll
                for (int i = 0; i < Q; ++i) mn[i] |= ((bc >> i) & 1u) << e;
            }
            wave_sync();  // the next cycle's table overwrites s_val
        }
#pragma unroll
        for (int i = 0; i < Q; ++i) m[i] = mn[i] & vm;
    }

    // layer format: planes s_i = sign(pa_i) b_i, exponents P_i.  Four sign
    // bits become four bytes (+1 = 0x01, -1 = 0xff): spread bit j to bit 8 j,
    // times 0xfe, xor 0xffffffff.
#pragma unroll
    for (int i = 0; i < Q; ++i) {
        const uint32_t bits = ((int8_t)(ps[i] & 0xffu) < 0 ? ~m[i] : m[i]);
        uint32_t word[E / 4 > 0 ? E / 4 : 1];
#pragma unroll
        for (int u = 0; u < E / 4; ++u) {
            const uint32_t nib = (bits >> (4 * u)) & 15u;
            word[u] = ~(((nib * 0x204081u) & 0x01010101u) * 0xfeu);
        }
        int8_t* dst = cs + i * plane + l * E;
        if constexpr (E == 2) {
            const uint32_t two = bits & 3u;
            *reinterpret_cast<uint16_t*>(dst) =
                (uint16_t)~(((two * 0x81u) & 0x0101u) * 0xfeu);
        } else if constexpr (E == 4) {
            *reinterpret_cast<uint32_t*>(dst) = word[0];
        } else {
#pragma unroll
            for (int u = 0; u < E / 8; ++u)
                if (FULL || l * E + 8 * u < G)
                    *reinterpret_cast<uint2*>(dst + 8 * u) = make_uint2(word[2 * u], word[2 * u + 1]);
        }
    }
    if (l == 0) write_scales<Q>(pe, ps, terms, ex, tsg, ex_plane);
}

// Each group of LN lanes walks the segments with a stride of the whole grid
// and loads the next segment's weights before working on the current one.
// The kernel is bound by fp64 VALU issue; at least two waves per SIMD (at
// most 256 VGPRs) measured faster than one wave with more registers.
template <int Q, int E, int LN, bool FULL>
__global__ __launch_bounds__(kQuantThreads, 2) void k_quantize_seg(
    const float* __restrict__ w, int N, int K, int G, int cycles, int terms,
    int8_t* __restrict__ signs, int8_t* __restrict__ exps, int8_t* __restrict__ tsg) {
    constexpr int kSegs = kQuantThreads / LN;
    __shared__ SegLds<Q, LN> lds;
    const int l = threadIdx.x & (LN - 1);
    const int sb = threadIdx.x / LN;
    const int NG = K / G;
    const int64_t total = (int64_t)N * NG;
    const int64_t stride = (int64_t)gridDim.x * kSegs;
    int64_t seg = (int64_t)blockIdx.x * kSegs + sb;
    if (seg >= total) return;  // all LN lanes of the group
    const int64_t plane = (int64_t)N * K;
    const int64_t ex_plane = total;

    float wn[E];
    auto load = [&](int64_t sg, float (&dst)[E]) {
        const int n = (int)(sg / NG), g = (int)(sg % NG);
        const float* ws = w + (int64_t)n * K + (int64_t)g * G + l * E;
        if constexpr (E == 2) {
            const float2 v = *reinterpret_cast<const float2*>(ws);
            dst[0] = v.x;
            dst[1] = v.y;
        } else {
#pragma unroll
            for (int u = 0; u < E / 4; ++u) {
                // runs of 8 slots are wholly valid or wholly empty
                const bool ok = FULL || l * E + 8 * (u / 2) < G;
                const float4 v = ok ? *reinterpret_cast<const float4*>(ws + 4 * u)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
                dst[4 * u] = v.x;
                dst[4 * u + 1] = v.y;
                dst[4 * u + 2] = v.z;
                dst[4 * u + 3] = v.w;
            }
        }
    };
    load(seg, wn);
    for (; seg < total; seg += stride) {
        float wf[E];
#pragma unroll
        for (int e = 0; e < E; ++e) wf[e] = wn[e];
        if (seg + stride < total) load(seg + stride, wn);
        const int n = (int)(seg / NG), g = (int)(seg % NG);
        const int64_t at = ((int64_t)n * NG + g) * terms;
        quantize_segment<Q, E, LN, FULL>(wf, l, sb, G, cycles, terms,
                                         signs + (int64_t)n * K + (int64_t)g * G, plane,
                                         exps + at, tsg ? tsg + at : nullptr, ex_plane, lds);
    }
}

struct QuantArgs {
    const float* w;
    int N, K, G, cycles, terms;
    int8_t* signs;
    int8_t* exps;
    int8_t* tsg;
    int64_t segs;
};

template <int Q, int E, int LN>
void launch_seg(const QuantArgs& a, hipStream_t s) {
    constexpr int kSegs = kQuantThreads / LN;
    const int64_t blocks = (a.segs + kSegs - 1) / kSegs;
    const unsigned grid = (unsigned)(blocks < kSegMaxBlocks ? blocks : kSegMaxBlocks);
    const bool full = E < 8 || a.G == LN * E;  // E < 8: only ever full (G = 8 or 16)
    if (full)
        hipLaunchKernelGGL((k_quantize_seg<Q, E, LN, true>), dim3(grid), dim3(kQuantThreads), 0,
                           s, a.w, a.N, a.K, a.G, a.cycles, a.terms, a.signs, a.exps, a.tsg);
    else if constexpr (E >= 8)
        hipLaunchKernelGGL((k_quantize_seg<Q, E, LN, false>), dim3(grid), dim3(kQuantThreads), 0,
                           s, a.w, a.N, a.K, a.G, a.cycles, a.terms, a.signs, a.exps, a.tsg);
}

// Lanes per segment and slots per lane.  q <= 4: 4 lanes up to G = 128 (E =
// G / 4 rounded up to a power of two, at least 8 when a run of slots can be
// empty), 8 lanes of 32 slots above.  q > 4 (the 2^q code values in LDS): 16
// lanes of 16 slots, 16 segments per workgroup.
template <int Q>
void launch_seg_e(const QuantArgs& a, hipStream_t s) {
    if constexpr (Q > 4) {
        launch_seg<Q, 16, 16>(a, s);
    } else {
        if (a.G == 8)
            launch_seg<Q, 2, 4>(a, s);
        else if (a.G == 16)
            launch_seg<Q, 4, 4>(a, s);
        else if (a.G <= 32)
            launch_seg<Q, 8, 4>(a, s);
        else if (a.G <= 64)
            launch_seg<Q, 16, 4>(a, s);
        else if (a.G <= 128)
            launch_seg<Q, 32, 4>(a, s);
        else
            launch_seg<Q, 32, 8>(a, s);
    }
}

template <int Q>
void launch_wave(const QuantArgs& a, hipStream_t s) {
    const unsigned grid = (unsigned)((a.segs + kWaves - 1) / kWaves);
    hipLaunchKernelGGL(k_quantize_bcq<Q>, dim3(grid), dim3(kQuantThreads), 0, s, a.w, a.N, a.K,
                       a.G, a.cycles, a.terms, a.signs, a.exps, a.tsg);
}

template <int Q>
void launch_q(const QuantArgs& a, hipStream_t s) {
    if (a.G <= kSegMaxGroup)
        launch_seg_e<Q>(a, s);
    else
        launch_wave<Q>(a, s);
}

int quantize(const float* w, int N, int K, int q, int group, int cycles, int terms,
             int8_t* signs, int8_t* exps, int8_t* tsg, void* stream) {
    if (!w || !signs || !exps) return SA_ERR_NULL;
    if (q < 1 || q > SA_MAX_Q) return SA_ERR_Q;
    if (N < 1 || K < 8 || (K & 7)) return SA_ERR_SHAPE;
    if ((int64_t)q * N * K > (int64_t)1 << 36) return SA_ERR_SHAPE;
    if ((int64_t)N * (K / 8) >= (int64_t)1 << 31) return SA_ERR_SHAPE;
    if (group < 8 || (group & 7) || (K % group)) return SA_ERR_GROUP;
    if (cycles < 0 || cycles > SA_MAX_CYCLES) return SA_ERR_SHAPE;
    if (terms < 1 || terms > SA_MAX_TERMS) return SA_ERR_SHAPE;
    if ((reinterpret_cast<uintptr_t>(w) & 15u) || (reinterpret_cast<uintptr_t>(signs) & 7u))
        return SA_ERR_ALIGN;
    QuantArgs a{w, N, K, group, cycles, terms, signs, exps, tsg, (int64_t)N * (K / group)};
    if ((a.segs + kWaves - 1) / kWaves > 0x7fffffff) return SA_ERR_SHAPE;
    const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    switch (q) {
        case 1: launch_q<1>(a, s); break;
        case 2: launch_q<2>(a, s); break;
        case 3: launch_q<3>(a, s); break;
        case 4: launch_q<4>(a, s); break;
        case 5: launch_q<5>(a, s); break;
        case 6: launch_q<6>(a, s); break;
        case 7: launch_q<7>(a, s); break;
        default: launch_q<8>(a, s); break;
    }
    return hipGetLastError() == hipSuccess ? SA_OK : SA_ERR_HIP;
}

}  // namespace

SA_API int sa_quantize_bcq(const float* w, int N, int K, int q, int group, int cycles,
                           int8_t* signs, int8_t* exps, void* stream) {
    return quantize(w, N, K, q, group, cycles, 1, signs, exps, nullptr, stream);
}

SA_API int sa_quantize_bcq_terms(const float* w, int N, int K, int q, int group, int cycles,
                                 int terms, int8_t* signs, int8_t* exps, int8_t* term_signs,
                                 void* stream) {
    if (!term_signs) return SA_ERR_NULL;
    return quantize(w, N, K, q, group, cycles, terms, signs, exps, term_signs, stream);
}
