// gfx950 kernels and C ABI of the shift-add linear layer (ShiftAddLLM, Sec. 4.1).
//
//   y[b][n] = sum_i sum_g 2^e[i][n][g] * sum_{k in g} s_i[n][k] x[b][k]
//
// computed as: 256-entry tables of signed partial sums per 8 activations
// (built in LDS), one table query per packed weight byte, fp32 adds, and one
// ldexp per (plane, row, 128-column block) folded into the fp32 accumulation.
// The path is an HBM stream of packed bits, not a dense contraction: no MFMA.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <map>
#include <mutex>
#include <utility>

#include "shiftadd.h"

#define SA_VERSION_STRING "0.1.0 gfx950"

namespace {

constexpr int kThreads = 256;     // 4 waves of 64
constexpr int kTileRows = 64;     // rows per tile: one row per lane
constexpr int kBlockChunks = 16;  // chunks (8 columns each) per block: 128 columns
constexpr int kKeyStride = 64;    // floats per key in the LDS tables (256 bytes)

__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }

// Byte offset of the key of (plane i, row n, chunk c) in the packed layout.
// Rows come in tiles of 64 and chunks in blocks of 16; a 64-row tile of one
// block is a contiguous piece, 16 bytes per row.  Inside a full block the 16
// keys of row r are rotated by r: position p holds chunk (p + r) mod 16, so
// that the lanes of a wave querying position p touch 16 different tables.
__host__ __device__ inline int64_t layout_offset(int i, int n, int c, int N, int C) {
    const int T = n >> 6, r = n & 63;
    const int R = imin(kTileRows, N - kTileRows * T);
    const int J = c >> 4, u = c & 15;
    const int U = imin(kBlockChunks, C - kBlockChunks * J);
    const int p = (U == kBlockChunks) ? ((u - r) & 15) : u;
    return ((int64_t)i * N + (int64_t)kTileRows * T) * C + (int64_t)kBlockChunks * J * R +
           (int64_t)r * U + p;
}

__device__ inline float half_bits_to_float(uint32_t h) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}

// The 8 activations x[8c..8c+7] of one chunk (16 bytes, 16-byte aligned).
__device__ inline void load_chunk(const uint16_t* p, float f[8]) {
    const uint4 v = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        f[2 * j] = half_bits_to_float(w[j] & 0xffffu);
        f[2 * j + 1] = half_bits_to_float(w[j] >> 16);
    }
}

// Signed sums of 4 activations for every 4-bit pattern a (bit j set -> +x_j):
// out[a] = (+-x0 +-x1) + (+-x2 +-x3).  Flipping every bit of a negates the
// result exactly, so table entries m and 255-m are exact negatives.
__device__ inline void nibble_sums(float x0, float x1, float x2, float x3, float out[16]) {
    const float p01[4] = {-x0 - x1, x0 - x1, x1 - x0, x0 + x1};
    const float p23[4] = {-x2 - x3, x2 - x3, x3 - x2, x2 + x3};
#pragma unroll
    for (int a = 0; a < 16; ++a) out[a] = p01[a & 3] + p23[a >> 2];
}

// One high-nibble sum (activations 4..7 of the chunk) for pattern h.
__device__ inline float nibble_sum(float x4, float x5, float x6, float x7, int h) {
    const float a = (h & 1) ? x4 : -x4;
    const float b = (h & 2) ? x5 : -x5;
    const float c = (h & 4) ? x6 : -x6;
    const float d = (h & 8) ? x7 : -x7;
    return (a + b) + (c + d);
}
// Table entry m of a chunk = low-nibble sum of (m & 15) + high-nibble sum of (m >> 4).

// ---------------------------------------------------------------- pack / unpack

__global__ void k_pack(const int8_t* __restrict__ signs, int q, int N, int C,
                       uint8_t* __restrict__ packed) {
    const int64_t total = (int64_t)q * N * C;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int c = (int)(t % C);
        const int64_t rest = t / C;
        const int n = (int)(rest % N);
        const int i = (int)(rest / N);
        const int8_t* s = signs + t * 8;
        uint32_t v = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) v |= (s[j] > 0 ? 1u : 0u) << j;
        packed[layout_offset(i, n, c, N, C)] = (uint8_t)v;
    }
}

__global__ void k_unpack(const uint8_t* __restrict__ packed, int q, int N, int C,
                         int8_t* __restrict__ signs) {
    const int64_t total = (int64_t)q * N * C;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int c = (int)(t % C);
        const int64_t rest = t / C;
        const int n = (int)(rest % N);
        const int i = (int)(rest / N);
        const uint32_t v = packed[layout_offset(i, n, c, N, C)];
        int8_t* s = signs + t * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = ((v >> j) & 1u) ? (int8_t)1 : (int8_t)-1;
    }
}

// ---------------------------------------------------------------- tables

// One item = (batch row b, chunk c, high nibble h): the 16 entries 16h..16h+15.
__global__ void k_build_lut(const uint16_t* __restrict__ x, int K, int B, float* __restrict__ lut) {
    const int C = K >> 3;
    const int64_t total = (int64_t)B * C * 16;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
        const int h = (int)(t & 15);
        const int64_t bc = t >> 4;  // b * C + c
        const int b = (int)(bc / C), c = (int)(bc % C);
        float f[8];
        load_chunk(x + (int64_t)b * K + 8 * c, f);
        float lo[16];
        nibble_sums(f[0], f[1], f[2], f[3], lo);
        const float hi = nibble_sum(f[4], f[5], f[6], f[7], h);
        float4* out = reinterpret_cast<float4*>(lut + bc * 256 + 16 * h);
#pragma unroll
        for (int a = 0; a < 4; ++a)
            out[a] = make_float4(lo[4 * a] + hi, lo[4 * a + 1] + hi, lo[4 * a + 2] + hi,
                                 lo[4 * a + 3] + hi);
    }
}

// ---------------------------------------------------------------- generic kernel
//
// Any group size (group % 8 == 0).  One workgroup = 256 output rows of one
// batch row; K is walked in blocks of 16 chunks whose tables are staged in LDS.
// Each row keeps one fp32 partial per plane (in LDS) across blocks and shifts it
// into its total when a group ends.
__global__ __launch_bounds__(kThreads) void k_gemm_generic(
    const uint16_t* __restrict__ x, const uint8_t* __restrict__ packed,
    const int8_t* __restrict__ exps, int q, int N, int K, int G, float* __restrict__ y) {
    __shared__ float lut[kBlockChunks][256];
    __shared__ float part[SA_MAX_Q][kThreads];
    const int C = K >> 3, NG = K / G, b = blockIdx.y;
    const int n = blockIdx.x * kThreads + threadIdx.x;
    const bool active = n < N;
    const uint16_t* xb = x + (int64_t)b * K;
    for (int i = 0; i < SA_MAX_Q; ++i) part[i][threadIdx.x] = 0.0f;
    float total = 0.0f;
    for (int J = 0; J * kBlockChunks < C; ++J) {
        const int U = imin(kBlockChunks, C - kBlockChunks * J);
        {
            const int u = threadIdx.x >> 4, h = threadIdx.x & 15;
            if (u < U) {
                float f[8];
                load_chunk(xb + 8 * (kBlockChunks * J + u), f);
                float lo[16];
                nibble_sums(f[0], f[1], f[2], f[3], lo);
                const float hi = nibble_sum(f[4], f[5], f[6], f[7], h);
#pragma unroll
                for (int a = 0; a < 16; ++a) lut[u][16 * h + a] = lo[a] + hi;
            }
        }
        __syncthreads();
        if (active) {
            for (int i = 0; i < q; ++i) {
                float acc = part[i][threadIdx.x];
                for (int u = 0; u < U; ++u) {
                    const int c = kBlockChunks * J + u;
                    acc += lut[u][packed[layout_offset(i, n, c, N, C)]];
                    if ((8 * (c + 1)) % G == 0) {
                        const int g = (8 * c) / G;
                        total += ldexpf(acc, (int)exps[((int64_t)i * N + n) * NG + g]);
                        acc = 0.0f;
                    }
                }
                part[i][threadIdx.x] = acc;
            }
        }
        __syncthreads();
    }
    if (active) y[(int64_t)b * N + n] = total;
}

// ---------------------------------------------------------------- split-K table kernel
//
// group % 128 == 0.  Workgroup (range, slice): output rows of `range` (tiles of
// 64 rows, one row per lane, one tile per wave at a time) against the
// 128*GB input columns of `slice` (GB blocks of 16 chunks).
//
// LDS tables: key m of table slot s (slot = 16*block + chunk within block) for
// batch row bb is the float at byte m*256 + 4*(s*BB + bb).  A lane queries with
// one v_perm_b32 that places its key byte in bits 8..15 and its slot offset in
// bits 0..7 of the address.  Lanes 16l..16l+15 query block (j + l) mod nb at
// step j, and, through the rotated packed layout, 16 different chunks of it at
// each position, so the 32 lanes of a half-wave read 32 different slots: 32
// different banks.
//
// Each lane adds 16 queried entries (one block of one plane), shifts the sum by
// the exponent of its (plane, row, group) with ldexp and accumulates in fp32.
// Slices of one row tile meet through a workspace: every wave writes its tile's
// partial sums, and the last of the k_slices waves to finish a tile (atomic
// ticket) adds them in slice order and writes y.  The order is fixed, so the
// result is deterministic.

struct SplitKArgs {
    const uint16_t* x;     // activations of this pass, rows b0..b0+nbr-1
    int x_stride;          // elements between batch rows (K)
    int nbr;               // batch rows in this pass (<= BB)
    const uint8_t* packed;
    const int8_t* exps;
    int q, N, K, G;
    float* y;              // output rows of this pass
    int y_stride;          // elements between batch rows (N)
    float* partials;       // [k_slices][BB][N]
    unsigned* tickets;     // [ceil(N/64)], zero between calls
    int k_slices, row_ranges, tiles_per_range;
};

template <int BB>
__device__ inline void query_add(const char* lut_bytes, uint32_t addr, float acc[BB]) {
    if constexpr (BB == 1) {
        acc[0] += *reinterpret_cast<const float*>(lut_bytes + addr);
    } else if constexpr (BB == 2) {
        const float2 v = *reinterpret_cast<const float2*>(lut_bytes + addr);
        acc[0] += v.x;
        acc[1] += v.y;
    } else {
        const float4 v = *reinterpret_cast<const float4*>(lut_bytes + addr);
        acc[0] += v.x;
        acc[1] += v.y;
        acc[2] += v.z;
        acc[3] += v.w;
    }
}

template <int GB, int BB>
__global__ __launch_bounds__(kThreads) void k_gemm_splitk(SplitKArgs a) {
    static_assert(kBlockChunks * GB * BB <= kKeyStride, "slot offsets must fit in one byte");
    __shared__ float lut[256 * kKeyStride];
    const int C = a.K >> 3, C16 = C >> 4, NG = a.K / a.G, bpg = a.G >> 7;

    // Workgroup -> (range, slice).  Workgroups are dispatched round-robin over
    // the 8 XCDs; when row_ranges % 8 == 0 every slice of a range lands on the
    // same XCD, so they share its L2 for exponents and partial sums.
    int range, slice;
    {
        const int w = blockIdx.x;
        if ((a.row_ranges & 7) == 0) {
            const int xcd = w & 7, u = w >> 3;
            slice = u % a.k_slices;
            range = ((u / a.k_slices) << 3) | xcd;
        } else {
            range = w / a.k_slices;
            slice = w % a.k_slices;
        }
    }
    const int J0 = slice * GB;
    const int nb = imin(GB, C16 - J0);
    const int ncol = kBlockChunks * nb * BB;

    // ---- tables for this slice: item (column, quarter of the high nibbles)
    for (int t = threadIdx.x; t < ncol * 4; t += kThreads) {
        const int col = t % ncol, hq = t / ncol;
        const int bb = col % BB, slot = col / BB;
        const int c = kBlockChunks * (J0 + (slot >> 4)) + (slot & 15);
        float f[8];
        if (bb < a.nbr) {
            load_chunk(a.x + (int64_t)bb * a.x_stride + 8 * c, f);
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) f[j] = 0.0f;
        }
        float lo[16];
        nibble_sums(f[0], f[1], f[2], f[3], lo);
#pragma unroll
        for (int hh = 0; hh < 4; ++hh) {
            const int h = 4 * hq + hh;
            const float hi = nibble_sum(f[4], f[5], f[6], f[7], h);
#pragma unroll
            for (int m = 0; m < 16; ++m) lut[(16 * h + m) * kKeyStride + col] = lo[m] + hi;
        }
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // Block of register slot j for this lane, and the slot offsets of its 16
    // positions (4 per register, one per byte).
    int blk[GB];
    uint32_t offs[GB][4];
#pragma unroll
    for (int j = 0; j < GB; ++j) {
        const int g = nb > 0 ? (j + (lane >> 4)) % nb : 0;
        blk[j] = J0 + g;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            uint32_t v = 0;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int p = 4 * k + t;
                const uint32_t s = (uint32_t)(kBlockChunks * g + ((p + lane) & 15));
                v |= (s * 4u * BB) << (8 * t);
            }
            offs[j][k] = v;
        }
    }
    const char* lut_bytes = reinterpret_cast<const char*>(lut);

    const int tiles = (a.N + kTileRows - 1) / kTileRows;
    const int T0 = range * a.tiles_per_range;
    const int T1 = imin(T0 + a.tiles_per_range, tiles);
    for (int T = T0 + wave; T < T1; T += kThreads / 64) {
        const int R = imin(kTileRows, a.N - kTileRows * T);
        const bool active = lane < R;
        const int n = kTileRows * T + lane;
        float tot[BB];
#pragma unroll
        for (int bb = 0; bb < BB; ++bb) tot[bb] = 0.0f;

        // all planes of this tile: keys and exponents
        uint4 wv[SA_MAX_Q][GB];
        int ev[SA_MAX_Q][GB];
#pragma unroll
        for (int i = 0; i < SA_MAX_Q; ++i) {
            if (i < a.q) {
                const uint8_t* base =
                    a.packed + ((int64_t)i * a.N + (int64_t)kTileRows * T) * C + 16 * lane;
                const int8_t* erow = a.exps + ((int64_t)i * a.N + n) * NG;
#pragma unroll
                for (int j = 0; j < GB; ++j) {
                    if (j < nb && active) {
                        wv[i][j] = *reinterpret_cast<const uint4*>(
                            base + (int64_t)kBlockChunks * blk[j] * R);
                        ev[i][j] = erow[blk[j] / bpg];
                    } else {
                        wv[i][j] = make_uint4(0, 0, 0, 0);
                        ev[i][j] = 0;
                    }
                }
            }
        }
#pragma unroll
        for (int i = 0; i < SA_MAX_Q; ++i) {
            if (i < a.q) {
#pragma unroll
                for (int j = 0; j < GB; ++j) {
                    if (j < nb) {
                        float acc[BB];
#pragma unroll
                        for (int bb = 0; bb < BB; ++bb) acc[bb] = 0.0f;
                        const uint32_t words[4] = {wv[i][j].x, wv[i][j].y, wv[i][j].z, wv[i][j].w};
#pragma unroll
                        for (int k = 0; k < 4; ++k) {
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                // byte 0: slot offset (offs byte t); byte 1: key (word byte t)
                                const uint32_t sel = 0x0c0c0000u | ((4u + t) << 8) | (uint32_t)t;
                                const uint32_t addr =
                                    __builtin_amdgcn_perm(words[k], offs[j][k], sel);
                                query_add<BB>(lut_bytes, addr, acc);
                            }
                        }
#pragma unroll
                        for (int bb = 0; bb < BB; ++bb) tot[bb] += ldexpf(acc[bb], ev[i][j]);
                    }
                }
            }
        }

        if (a.k_slices == 1) {
            if (active)
                for (int bb = 0; bb < a.nbr; ++bb) a.y[(int64_t)bb * a.y_stride + n] = tot[bb];
            continue;
        }
        if (active)
            for (int bb = 0; bb < a.nbr; ++bb)
                a.partials[((int64_t)slice * BB + bb) * a.N + n] = tot[bb];
        __threadfence();
        unsigned ticket = 0;
        if (lane == 0) ticket = atomicAdd(&a.tickets[T], 1u);
        ticket = __shfl(ticket, 0);
        if (ticket == (unsigned)(a.k_slices - 1)) {
            __threadfence();
            if (active) {
                for (int bb = 0; bb < a.nbr; ++bb) {
                    const float* src = a.partials + (int64_t)bb * a.N + n;
                    float s = 0.0f;
                    for (int sl = 0; sl < a.k_slices; ++sl)
                        s += __builtin_nontemporal_load(src + (int64_t)sl * BB * a.N);
                    a.y[(int64_t)bb * a.y_stride + n] = s;
                }
            }
            if (lane == 0) atomicExch(&a.tickets[T], 0u);
        }
    }
}

// ---------------------------------------------------------------- host side

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_dims(int q, int N, int K) {
    if (q < 1 || q > SA_MAX_Q) return SA_ERR_Q;
    if (N < 1 || K < 8 || (K & 7)) return SA_ERR_SHAPE;
    // every element count that the kernels index must fit comfortably
    if ((int64_t)q * N * K > (int64_t)1 << 36) return SA_ERR_SHAPE;
    return SA_OK;
}

int validate_gemm(const void* x, const void* packed, const void* exps, int q, int N, int K,
                  int group, int batch, const void* y) {
    if (!x || !packed || !exps || !y) return SA_ERR_NULL;
    int st = check_dims(q, N, K);
    if (st != SA_OK) return st;
    if (batch < 1 || batch > SA_MAX_BATCH) return SA_ERR_SHAPE;
    if (group < 8 || (group & 7) || (K % group)) return SA_ERR_GROUP;
    if (!aligned16(x) || !aligned16(packed) || !aligned16(y)) return SA_ERR_ALIGN;
    return SA_OK;
}

struct PassShape {
    int gb, bb;
};

PassShape pass_shape(int rem) {
    if (rem >= 3) return {1, 4};
    if (rem == 2) return {2, 2};
    return {2, 1};
}

void make_plan(int q, int N, int K, int group, int batch, sa_plan* p) {
    *p = sa_plan{};
    p->threads = kThreads;
    const int tiles = (N + kTileRows - 1) / kTileRows;
    if (group % 128 != 0) {
        p->path = 0;
        p->blocks_per_slice = (K / 8 + kBlockChunks - 1) / kBlockChunks;
        p->batch_per_pass = 1;
        p->passes = 1;
        p->k_slices = 1;
        p->row_ranges = (N + kThreads - 1) / kThreads;
        p->rows_per_range = kThreads;
        p->workgroups = p->row_ranges * batch;
        p->lds_bytes = sizeof(float) * (kBlockChunks * 256 + SA_MAX_Q * kThreads);
        p->workspace_bytes = 0;
        return;
    }
    const PassShape first = pass_shape(batch);
    p->path = 1;
    p->blocks_per_slice = first.gb;
    p->batch_per_pass = first.bb;
    int passes = 0, rem = batch;
    while (rem > 0) {
        rem -= imin(rem, pass_shape(rem).bb);
        ++passes;
    }
    p->passes = passes;
    const int C16 = K / 128;
    const int k_slices = (C16 + first.gb - 1) / first.gb;
    const int waves = kThreads / 64;
    const int ranges0 = (tiles + waves - 1) / waves;
    // Give a workgroup more tiles (re-using its tables) once the grid would
    // exceed ~2 workgroups per CU.
    int per = (int)(((int64_t)ranges0 * k_slices) / 512);
    if (per < 1) per = 1;
    const int tiles_per_range = waves * per;
    const int row_ranges = (tiles + tiles_per_range - 1) / tiles_per_range;
    p->k_slices = k_slices;
    p->row_ranges = row_ranges;
    p->rows_per_range = tiles_per_range * kTileRows;
    p->workgroups = row_ranges * k_slices;
    p->lds_bytes = sizeof(float) * 256 * kKeyStride;
    if (k_slices > 1)
        p->workspace_bytes =
            sizeof(unsigned) * (size_t)tiles + sizeof(float) * (size_t)k_slices * first.bb * N;
}

// Split-K workspace per (device, stream): a ticket array (one counter per
// 64-row tile) and a partial-sum array, in separate buffers.  Tickets are
// zeroed when their buffer is allocated and every call leaves them at zero;
// nothing else is ever written to the ticket buffer.
struct Workspace {
    unsigned* tickets = nullptr;
    size_t ticket_count = 0;
    float* partials = nullptr;
    size_t partial_bytes = 0;
};
std::mutex g_mu;
std::map<std::pair<int, void*>, Workspace> g_ws;

int get_workspace(void* stream, size_t tickets, size_t partial_bytes, unsigned** t_out,
                  float** p_out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return SA_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    Workspace& w = g_ws[{dev, stream}];
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool grow_t = w.ticket_count < tickets, grow_p = w.partial_bytes < partial_bytes;
    if ((grow_t && w.tickets) || (grow_p && w.partials)) {
        if (hipStreamSynchronize(s) != hipSuccess) return SA_ERR_HIP;
    }
    if (grow_t) {
        if (w.tickets) (void)hipFree(w.tickets);
        w.tickets = nullptr;
        w.ticket_count = 0;
        size_t want = tickets < 4096 ? 4096 : tickets;
        void* p = nullptr;
        if (hipMalloc(&p, want * sizeof(unsigned)) != hipSuccess) return SA_ERR_NOMEM;
        if (hipMemsetAsync(p, 0, want * sizeof(unsigned), s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            (void)hipFree(p);
            return SA_ERR_HIP;
        }
        w.tickets = static_cast<unsigned*>(p);
        w.ticket_count = want;
    }
    if (grow_p) {
        if (w.partials) (void)hipFree(w.partials);
        w.partials = nullptr;
        w.partial_bytes = 0;
        size_t want = partial_bytes < ((size_t)1 << 20) ? ((size_t)1 << 20) : partial_bytes;
        void* p = nullptr;
        if (hipMalloc(&p, want) != hipSuccess) return SA_ERR_NOMEM;
        w.partials = static_cast<float*>(p);
        w.partial_bytes = want;
    }
    *t_out = w.tickets;
    *p_out = w.partials;
    return SA_OK;
}

int launch_status() { return hipGetLastError() == hipSuccess ? SA_OK : SA_ERR_HIP; }

int grid_for(int64_t items) {
    int64_t g = (items + kThreads - 1) / kThreads;
    if (g > 16384) g = 16384;
    if (g < 1) g = 1;
    return (int)g;
}

template <int GB, int BB>
void launch_splitk(const SplitKArgs& a, int workgroups, hipStream_t s) {
    hipLaunchKernelGGL((k_gemm_splitk<GB, BB>), dim3(workgroups), dim3(kThreads), 0, s, a);
}

}  // namespace

extern "C" {

SA_API size_t sa_packed_bytes(int q, int N, int K) {
    if (check_dims(q, N, K) != SA_OK) return 0;
    return (size_t)q * N * (K / 8);
}

SA_API int64_t sa_packed_offset(int q, int N, int K, int i, int n, int c) {
    if (check_dims(q, N, K) != SA_OK) return -1;
    if (i < 0 || i >= q || n < 0 || n >= N || c < 0 || c >= K / 8) return -1;
    return layout_offset(i, n, c, N, K / 8);
}

SA_API int sa_pack_weights(const int8_t* signs, int q, int N, int K, uint8_t* packed_bits,
                           void* stream) {
    if (!signs || !packed_bits) return SA_ERR_NULL;
    const int st = check_dims(q, N, K);
    if (st != SA_OK) return st;
    if (!aligned16(packed_bits)) return SA_ERR_ALIGN;
    const int64_t items = (int64_t)q * N * (K / 8);
    hipLaunchKernelGGL(k_pack, dim3(grid_for(items)), dim3(kThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), signs, q, N, K / 8, packed_bits);
    return launch_status();
}

SA_API int sa_unpack_weights(const uint8_t* packed_bits, int q, int N, int K, int8_t* signs,
                             void* stream) {
    if (!signs || !packed_bits) return SA_ERR_NULL;
    const int st = check_dims(q, N, K);
    if (st != SA_OK) return st;
    if (!aligned16(packed_bits)) return SA_ERR_ALIGN;
    const int64_t items = (int64_t)q * N * (K / 8);
    hipLaunchKernelGGL(k_unpack, dim3(grid_for(items)), dim3(kThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), packed_bits, q, N, K / 8, signs);
    return launch_status();
}

SA_API int sa_build_lut(const uint16_t* x, int K, int batch, float* lut, void* stream) {
    if (!x || !lut) return SA_ERR_NULL;
    if (K < 8 || (K & 7) || batch < 1 || batch > SA_MAX_BATCH) return SA_ERR_SHAPE;
    if (!aligned16(x) || !aligned16(lut)) return SA_ERR_ALIGN;
    const int64_t items = (int64_t)batch * (K / 8) * 16;
    hipLaunchKernelGGL(k_build_lut, dim3(grid_for(items)), dim3(kThreads), 0,
                       reinterpret_cast<hipStream_t>(stream), x, K, batch, lut);
    return launch_status();
}

SA_API int sa_plan_gemm(int q, int N, int K, int group, int batch, sa_plan* plan) {
    if (!plan) return SA_ERR_NULL;
    int st = check_dims(q, N, K);
    if (st != SA_OK) return st;
    if (batch < 1 || batch > SA_MAX_BATCH) return SA_ERR_SHAPE;
    if (group < 8 || (group & 7) || (K % group)) return SA_ERR_GROUP;
    make_plan(q, N, K, group, batch, plan);
    return SA_OK;
}

SA_API int sa_shiftadd_gemm(const uint16_t* x, const uint8_t* packed_bits, const int8_t* exps,
                            int q, int N, int K, int group, int batch, float* y, void* stream) {
    const int st = validate_gemm(x, packed_bits, exps, q, N, K, group, batch, y);
    if (st != SA_OK) return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    sa_plan plan;
    make_plan(q, N, K, group, batch, &plan);
    if (plan.path == 0) {
        hipLaunchKernelGGL(k_gemm_generic, dim3(plan.row_ranges, batch), dim3(kThreads), 0, s,
                           x, packed_bits, exps, q, N, K, group, y);
        return launch_status();
    }
    const int tiles = (N + kTileRows - 1) / kTileRows;
    unsigned* tickets = nullptr;
    float* partials = nullptr;
    if (plan.workspace_bytes > 0) {
        const size_t pbytes = plan.workspace_bytes - sizeof(unsigned) * (size_t)tiles;
        const int wst = get_workspace(stream, (size_t)tiles, pbytes, &tickets, &partials);
        if (wst != SA_OK) return wst;
    }
    SplitKArgs a{};
    a.x_stride = K;
    a.packed = packed_bits;
    a.exps = exps;
    a.q = q;
    a.N = N;
    a.K = K;
    a.G = group;
    a.y_stride = N;
    a.tickets = tickets;
    a.partials = partials;
    a.row_ranges = plan.row_ranges;
    a.tiles_per_range = plan.rows_per_range / kTileRows;
    for (int b0 = 0; b0 < batch;) {
        const PassShape ps = pass_shape(batch - b0);
        const int nbr = imin(ps.bb, batch - b0);
        a.x = x + (int64_t)b0 * K;
        a.y = y + (int64_t)b0 * N;
        a.nbr = nbr;
        a.k_slices = (K / 128 + ps.gb - 1) / ps.gb;
        const int wgs = plan.row_ranges * a.k_slices;
        if (ps.bb == 4)
            launch_splitk<1, 4>(a, wgs, s);
        else if (ps.bb == 2)
            launch_splitk<2, 2>(a, wgs, s);
        else
            launch_splitk<2, 1>(a, wgs, s);
        const int lst = launch_status();
        if (lst != SA_OK) return lst;
        b0 += nbr;
    }
    return SA_OK;
}

SA_API const char* sa_status_string(int status) {
    switch (status) {
        case SA_OK: return "ok";
        case SA_ERR_NULL: return "a required pointer is NULL";
        case SA_ERR_SHAPE: return "invalid shape (N, K, batch or sizes out of range, or K % 8 != 0)";
        case SA_ERR_Q: return "q must be in [1, 8]";
        case SA_ERR_GROUP: return "group must be a multiple of 8 that divides K";
        case SA_ERR_ALIGN: return "x, packed_bits, y and lut must be 16-byte aligned";
        case SA_ERR_HIP: return "HIP runtime error or kernel launch failure";
        case SA_ERR_NOMEM: return "could not allocate the split-K workspace";
        default: return "unknown status";
    }
}

SA_API const char* sa_version(void) { return SA_VERSION_STRING; }

SA_API void sa_shutdown(void) {
    std::lock_guard<std::mutex> lock(g_mu);
    int cur = 0;
    (void)hipGetDevice(&cur);
    for (auto& kv : g_ws) {
        (void)hipSetDevice(kv.first.first);
        (void)hipStreamSynchronize(reinterpret_cast<hipStream_t>(kv.first.second));
        if (kv.second.tickets) (void)hipFree(kv.second.tickets);
        if (kv.second.partials) (void)hipFree(kv.second.partials);
    }
    (void)hipSetDevice(cur);
    g_ws.clear();
}

}  // extern "C"
