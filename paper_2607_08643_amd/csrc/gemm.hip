// Fused decode-GEMM for M tokens: Y = X W_hat^T + (X A^T) B^T.
//
// Each block owns BN = 64 weight rows and up to 128 tokens. For every K step
// of 64 inputs it decodes the 64 x 64 weight tile from the code and gain
// planes into LDS as bf16 (stage terms summed by the fmaf chain of the
// decoder assembly, protected columns taken from the int8 payload, so the
// tile is W_hat rounded to bf16), stages the X tile in LDS, and runs
// v_mfma_f32_16x16x32_bf16 on it. The weight tile is decoded once per token
// tile, so the decode cost per weight falls as M grows. LoRA is added in the
// epilogue from T = X A^T, computed by a small prep kernel.
#include "bsq_internal.h"

namespace bsq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int BN = 64;       // weight rows per block
constexpr int BK = 64;       // inputs per K step
constexpr int LDS_PAD = 8;   // bf16 padding per LDS row (breaks bank aliasing)
constexpr int LDK = BK + LDS_PAD;
constexpr int MAX_BM = 128;  // tokens per block

struct GemmArgs {
    const void *codes[BSQ_MAX_STAGES];
    const uint16_t *gains[BSQ_MAX_STAGES];
    const float *tab32[BSQ_MAX_STAGES];
    const int32_t *idx;
    const int8_t *q8;
    const float *scale;
    const uint16_t *X;
    const uint16_t *B;  // LoRA B [d_out][rank]
    const float *T;     // LoRA X A^T [M][16]
    int rank;
    int64_t M, ldx, d_out, d_in, pitch, C, k, words, ldy;
    void *Y;
    int y_bf16;
};

__device__ __forceinline__ int find_pos(const int32_t *idx, int64_t k, int32_t j)
{
    int64_t lo = 0, hi = k - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (idx[mid] < j) lo = mid + 1;
        else hi = mid;
    }
    return int(lo);
}

// T[m][r] = sum_j X[m][j] A[r][j], fp32. One block per (token, rank row).
__global__ __launch_bounds__(256) void gemm_lora_prep(const uint16_t *X, int64_t ldx, const uint16_t *A,
                                                      int rank, int64_t d_in, float *T)
{
    __shared__ float red[256];
    const int64_t m = blockIdx.x / BSQ_MAX_LORA_RANK;
    const int r = blockIdx.x % BSQ_MAX_LORA_RANK;
    const int t = threadIdx.x;
    float acc = 0.0f;
    if (r < rank)
        for (int64_t j = t; j < d_in; j += 256)
            acc = __builtin_fmaf(bf16_to_f32(X[m * ldx + j]), bf16_to_f32(A[int64_t(r) * d_in + j]), acc);
    red[t] = acc;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (t < o) red[t] += red[t + o];
        __syncthreads();
    }
    if (t == 0) T[m * BSQ_MAX_LORA_RANK + r] = (r < rank) ? red[0] : 0.0f;
}

template <int D, int S, int MT>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs a)
{
    constexpr int BM = 16 * MT;
    constexpr int CPR = BK / D;             // chunks per tile row per K step
    constexpr int NCH = BN * CPR;           // chunks per tile
    __shared__ __attribute__((aligned(16))) uint16_t s_w[BN * LDK];
    __shared__ __attribute__((aligned(16))) uint16_t s_x[BM * LDK];
    extern __shared__ uint32_t s_dyn[];     // protected bitmap [words], then fp32 tables (D == 8)
    uint32_t *s_bits = s_dyn;
    float *s_tab = reinterpret_cast<float *>(s_dyn + ((a.words + 3) & ~int64_t(3)));

    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    const int64_t n0 = int64_t(blockIdx.x) * BN;
    const int64_t m0 = int64_t(blockIdx.y) * BM;

    if (a.k > 0) {
        for (int64_t w = t; w < a.words; w += 256) s_bits[w] = 0u;
        __syncthreads();
        for (int64_t p = t; p < a.k; p += 256) {
            const int32_t j = a.idx[p];
            if (j >= 0 && j < a.d_in) atomicOr(&s_bits[j >> 5], 1u << (j & 31));
        }
    }
    if constexpr (D == 8) {
        for (int e = t; e < S * 256 * 8; e += 256) {
            const int s = e / (256 * 8);
            s_tab[e] = a.tab32[s][e - s * 256 * 8];
        }
    }
    __syncthreads();

    f32x4_t acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    for (int64_t k0 = 0; k0 < a.d_in; k0 += BK) {
        // X tile: BM x BK bf16, 8 elements per 16-byte load
        for (int e = t; e < BM * (BK / 8); e += 256) {
            const int r = e / (BK / 8), c8 = (e - r * (BK / 8)) * 8;
            const int64_t row = m0 + r, col = k0 + c8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (row < a.M && col < a.d_in) v = *reinterpret_cast<const uint4 *>(a.X + row * a.ldx + col);
            *reinterpret_cast<uint4 *>(s_x + r * LDK + c8) = v;
        }
        // weight tile: decode BN rows x CPR chunks
        for (int e = t; e < NCH; e += 256) {
            const int r = e / CPR, cc = e - r * CPR;
            const int64_t row = n0 + r;
            const int64_t c = k0 / D + cc;
            float v[D];
#pragma unroll
            for (int j = 0; j < D; ++j) v[j] = 0.0f;
            if (row < a.d_out && c < a.C) {
                const int64_t off = tile_index(row, c, a.pitch);
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    const uint32_t code = (D == 8) ? uint32_t(static_cast<const uint8_t *>(a.codes[s])[off])
                                                   : uint32_t(static_cast<const uint16_t *>(a.codes[s])[off]);
                    const float g = f16_bits_to_f32(a.gains[s][off]);
                    const float *y = (D == 8) ? (s_tab + (s * 256 + code) * 8) : (a.tab32[s] + size_t(code) * D);
                    const float4 *y4 = reinterpret_cast<const float4 *>(y);
#pragma unroll
                    for (int q = 0; q < D / 4; ++q) {
                        const float4 yy = y4[q];
                        v[4 * q + 0] = __builtin_fmaf(g, yy.x, v[4 * q + 0]);
                        v[4 * q + 1] = __builtin_fmaf(g, yy.y, v[4 * q + 1]);
                        v[4 * q + 2] = __builtin_fmaf(g, yy.z, v[4 * q + 2]);
                        v[4 * q + 3] = __builtin_fmaf(g, yy.w, v[4 * q + 3]);
                    }
                }
                if (a.k > 0) {
                    const int64_t col0 = c * D;
                    const uint32_t pm = (s_bits[col0 >> 5] >> (col0 & 31)) & ((1u << D) - 1u);
                    if (pm) {
#pragma unroll
                        for (int j = 0; j < D; ++j) {
                            if (!((pm >> j) & 1u)) continue;
                            const int p = find_pos(a.idx, a.k, int32_t(col0 + j));
                            v[j] = float(a.q8[row * q8_pitch(a.k) + p]) * a.scale[p];
                        }
                    }
                }
            }
            uint16_t h[D];
#pragma unroll
            for (int j = 0; j < D; ++j) h[j] = f32_to_bf16(v[j]);
            uint16_t *dst = s_w + r * LDK + cc * D;
#pragma unroll
            for (int q = 0; q < D / 8; ++q) reinterpret_cast<uint4 *>(dst)[q] = reinterpret_cast<const uint4 *>(h)[q];
        }
        __syncthreads();
        // MFMA: wave w owns weight rows [16w, 16w + 16) of the tile, all BM tokens.
        // A = X (16 tokens x 32 inputs), B = W_hat^T (32 inputs x 16 weight rows);
        // both operands take inputs [8*(lane/16), +8) of the 32, so any fixed
        // ordering of the K lanes inside the instruction cancels out.
#pragma unroll
        for (int kk = 0; kk < BK; kk += 32) {
            const int kq = kk + 8 * (lane >> 4);
            const uint4 bw = *reinterpret_cast<const uint4 *>(s_w + (16 * wave + (lane & 15)) * LDK + kq);
            const bf16x8_t bop = __builtin_bit_cast(bf16x8_t, bw);
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const uint4 ax = *reinterpret_cast<const uint4 *>(s_x + (16 * i + (lane & 15)) * LDK + kq);
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ax), bop, acc[i], 0, 0, 0);
            }
        }
        __syncthreads();
    }

    // epilogue: D[i][j] with token i = 4*(lane/16) + r, weight row j = lane % 16
    const int64_t n = n0 + 16 * wave + (lane & 15);
    if (n >= a.d_out) return;
    float bl[BSQ_MAX_LORA_RANK];
#pragma unroll
    for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) bl[q] = (q < a.rank) ? bf16_to_f32(a.B[n * a.rank + q]) : 0.0f;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t m = m0 + 16 * i + 4 * (lane >> 4) + r;
            if (m >= a.M) continue;
            float v = acc[i][r];
            if (a.rank > 0) {
                const float *Tm = a.T + m * BSQ_MAX_LORA_RANK;
#pragma unroll
                for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) v = __builtin_fmaf(bl[q], Tm[q], v);
            }
            if (a.y_bf16) static_cast<uint16_t *>(a.Y)[m * a.ldy + n] = f32_to_bf16(v);
            else static_cast<float *>(a.Y)[m * a.ldy + n] = v;
        }
    }
}

template <int D, int S>
hipError_t launch_gemm_t(const GemmArgs &a, hipStream_t st)
{
    const int64_t nb = (a.d_out + BN - 1) / BN;
    const size_t shm = size_t((a.words + 3) & ~int64_t(3)) * 4 + ((D == 8) ? size_t(S) * 256 * 8 * 4 : 0);
    if (a.M <= 16) {
        hipLaunchKernelGGL((gemm_kernel<D, S, 1>), dim3(unsigned(nb), unsigned((a.M + 15) / 16)), dim3(256), shm, st, a);
    } else if (a.M <= 64) {
        hipLaunchKernelGGL((gemm_kernel<D, S, 4>), dim3(unsigned(nb), unsigned((a.M + 63) / 64)), dim3(256), shm, st, a);
    } else {
        hipLaunchKernelGGL((gemm_kernel<D, S, 8>), dim3(unsigned(nb), unsigned((a.M + MAX_BM - 1) / MAX_BM)), dim3(256),
                           shm, st, a);
    }
    return hipGetLastError();
}

}  // namespace

size_t gemm_ws_bytes(const bsq_config &cfg, int64_t d_in, int64_t M)
{
    (void)cfg;
    (void)d_in;
    return align256(size_t(M > 0 ? M : 1) * BSQ_MAX_LORA_RANK * 4);
}

hipError_t launch_gemm(const bsq_config &cfg, const void *codec, const bsq_layer &L, const bsq_lora *lora,
                       const void *X, int64_t M, int64_t ldx, void *Y, int y_dtype, int64_t ldy, void *ws,
                       hipStream_t st)
{
    GemmArgs a{};
    const char *cb = static_cast<const char *>(codec);
    for (int s = 0; s < cfg.stages; ++s) {
        a.codes[s] = L.codes[s];
        a.gains[s] = L.gains[s];
        a.tab32[s] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, s));
    }
    a.idx = L.prot_idx;
    a.q8 = L.prot_q8;
    a.scale = L.prot_scale;
    a.X = static_cast<const uint16_t *>(X);
    a.M = M;
    a.ldx = ldx;
    a.d_out = L.d_out;
    a.d_in = L.d_in;
    a.pitch = L.pitch;
    a.C = L.d_in / cfg.d;
    a.k = L.k;
    a.words = (L.k > 0) ? (L.d_in + 31) / 32 : 0;
    a.ldy = ldy;
    a.Y = Y;
    a.y_bf16 = (y_dtype == BSQ_BF16);
    a.rank = 0;
    a.T = static_cast<const float *>(ws);
    if (M == 0 || L.d_out == 0) return hipSuccess;
    if (lora && lora->rank > 0) {
        a.rank = lora->rank;
        a.B = lora->B;
        hipLaunchKernelGGL(gemm_lora_prep, dim3(unsigned(M * BSQ_MAX_LORA_RANK)), dim3(256), 0, st, a.X, ldx, lora->A,
                           lora->rank, L.d_in, static_cast<float *>(ws));
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int S = cfg.stages;
    if (cfg.d == 8) {
        switch (S) {
        case 1: return launch_gemm_t<8, 1>(a, st);
        case 2: return launch_gemm_t<8, 2>(a, st);
        case 3: return launch_gemm_t<8, 3>(a, st);
        default: return launch_gemm_t<8, 4>(a, st);
        }
    }
    switch (S) {
    case 1: return launch_gemm_t<16, 1>(a, st);
    case 2: return launch_gemm_t<16, 2>(a, st);
    case 3: return launch_gemm_t<16, 3>(a, st);
    default: return launch_gemm_t<16, 4>(a, st);
    }
}

}  // namespace bsq
