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

constexpr int BN = 64;       // weight rows per block (one 64-row group)
constexpr int BK = 128;      // inputs per K step
constexpr int LDS_PAD = 8;   // bf16 padding per LDS row (breaks bank aliasing)
constexpr int LDK = BK + LDS_PAD;

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

// Decode of one K step of the weight tile: rows [0, 64) of the 64-row group,
// the tile's chunks [cbeg, cbeg + CPS) (d = 8: all 16; d = 16: half), as
// bf16 into s_w. Thread t owns row t / 4 and CPT = CPS / 4 consecutive
// chunks; its code and gain words come from the prefetch registers.
template <int D, int S>
struct DecodeRegs {
    static constexpr int CPT = (D == 8) ? 4 : 2;     // chunks per thread per K step
    uint32_t code[S][(D == 8) ? 1 : 1];              // CPT codes: 4 bytes (d = 8) or 2 x uint16 (d = 16)
    uint32_t gain[S][CPT / 2];                        // CPT fp16 gains
};

template <int D, int S>
__device__ __forceinline__ void gemm_prefetch(DecodeRegs<D, S> &r, const GemmArgs &a, int64_t tile, int cbeg, int t)
{
    constexpr int CPT = DecodeRegs<D, S>::CPT;
    const int64_t e = (tile << 10) + ((t >> 2) << 4) + cbeg + (t & 3) * CPT;  // first element
#pragma unroll
    for (int s = 0; s < S; ++s) {
        if constexpr (D == 8) r.code[s][0] = *reinterpret_cast<const uint32_t *>(static_cast<const uint8_t *>(a.codes[s]) + e);
        else r.code[s][0] = *reinterpret_cast<const uint32_t *>(static_cast<const uint16_t *>(a.codes[s]) + e);
        if constexpr (CPT == 4) {
            const uint2 g = *reinterpret_cast<const uint2 *>(a.gains[s] + e);
            r.gain[s][0] = g.x;
            r.gain[s][1] = g.y;
        } else {
            r.gain[s][0] = *reinterpret_cast<const uint32_t *>(a.gains[s] + e);
        }
    }
}

template <int D, int S>
__device__ __forceinline__ void gemm_decode(const DecodeRegs<D, S> &r, const GemmArgs &a, const float *s_tab,
                                            const uint32_t *s_bits, uint16_t *s_w, int64_t rg, int64_t c0, int t)
{
    constexpr int CPT = DecodeRegs<D, S>::CPT;
    const int rr = t >> 2;
    const int64_t row = rg * 64 + rr;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
        const int64_t c = c0 + (t & 3) * CPT + u;  // chunk index in the row
        float v[D];
#pragma unroll
        for (int j = 0; j < D; ++j) v[j] = 0.0f;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint32_t code = (D == 8) ? ((r.code[s][0] >> (8 * u)) & 0xffu) : ((r.code[s][0] >> (16 * u)) & 0xffffu);
            const uint32_t gw = r.gain[s][u >> 1];
            const float g = f16_bits_to_f32(uint16_t((u & 1) ? (gw >> 16) : (gw & 0xffffu)));
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
        if (a.k > 0 && row < a.d_out && c < a.C) {
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
        uint16_t h[D];
#pragma unroll
        for (int j = 0; j < D; ++j) h[j] = f32_to_bf16(v[j]);
        uint16_t *dst = s_w + rr * LDK + ((t & 3) * CPT + u) * D;
#pragma unroll
        for (int q = 0; q < D / 8; ++q) reinterpret_cast<uint4 *>(dst)[q] = reinterpret_cast<const uint4 *>(h)[q];
    }
}

// One workgroup: the 64 rows of one row group x BM = WM * MT * 16 tokens.
// Waves are WM (token) x WN (row) with WM * WN = 4; a wave owns MT token
// groups and NT = 4 / WN row groups of 16. K steps of BK = 128 inputs.
template <int D, int S, int WM, int MT>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs a)
{
    constexpr int WN = 4 / WM, NT = 4 / WN, BM = WM * MT * 16;
    constexpr int CPS = BK / D;  // chunks per K step
    __shared__ __attribute__((aligned(16))) uint16_t s_w[BN * LDK];
    extern __shared__ uint32_t s_dyn[];  // protected bitmap [words], then fp32 tables (D == 8)
    uint32_t *s_bits = s_dyn;
    float *s_tab = reinterpret_cast<float *>(s_dyn + ((a.words + 3) & ~int64_t(3)));

    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int wm = wave % WM, wn = wave / WM;
    const int64_t rg = blockIdx.x;                        // row group
    const int64_t m0 = int64_t(blockIdx.y) * BM + wm * MT * 16;  // this wave's first token
    const int64_t nb = a.pitch / 16;                      // tiles per row group
    const int64_t ksteps = (a.C + CPS - 1) / CPS;         // K steps over the real chunks

    DecodeRegs<D, S> pre;
    gemm_prefetch<D, S>(pre, a, rg * nb, 0, t);
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

    f32x4_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // X fragments of a K step: token 16 i + lane % 16 of this wave, inputs
    // k0 + 32 kk4 + 8 (lane / 16) .. + 8. Loads are unconditional with the
    // token and input clamped into X (a clamped token's outputs are never
    // stored; a clamped input meets a zero weight), so they are not waited on
    // until the MFMAs need them, one K step later.
    uint4 xf[MT][BK / 32], xn[MT][BK / 32];
    auto load_x = [&](uint4 (&dst)[MT][BK / 32], int64_t k0) {
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            int64_t tok = m0 + 16 * i + (lane & 15);
            tok = tok < a.M ? tok : a.M - 1;
#pragma unroll
            for (int q = 0; q < BK / 32; ++q) {
                int64_t kq = k0 + 32 * q + 8 * (lane >> 4);
                kq = kq < a.d_in ? kq : a.d_in - 8;
                dst[i][q] = *reinterpret_cast<const uint4 *>(a.X + tok * a.ldx + kq);
            }
        }
    };
    load_x(xf, 0);

    for (int64_t ks = 0; ks < ksteps; ++ks) {
        const int64_t c0 = ks * CPS;  // first chunk of this step
        gemm_decode<D, S>(pre, a, s_tab, s_bits, s_w, rg, c0, t);
        const int64_t c1 = (ks + 1 < ksteps) ? c0 + CPS : c0;  // the last step reloads its own words
        gemm_prefetch<D, S>(pre, a, rg * nb + c1 / 16, int(c1 % 16), t);
        load_x(xn, c1 * D);
        __syncthreads();
#pragma unroll
        for (int q = 0; q < BK / 32; ++q) {
            bf16x8_t bop[NT];
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const uint4 bw = *reinterpret_cast<const uint4 *>(s_w + (16 * (wn * NT + j) + (lane & 15)) * LDK +
                                                                 32 * q + 8 * (lane >> 4));
                bop[j] = __builtin_bit_cast(bf16x8_t, bw);
            }
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const bf16x8_t aop = __builtin_bit_cast(bf16x8_t, xf[i][q]);
#pragma unroll
                for (int j = 0; j < NT; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, bop[j], acc[i][j], 0, 0, 0);
            }
        }
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int q = 0; q < BK / 32; ++q) xf[i][q] = xn[i][q];
        __syncthreads();
    }

    // epilogue: acc[i][j] element r is token 16 i + 4 (lane / 16) + r, row 16 j + lane % 16
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int64_t n = rg * 64 + 16 * (wn * NT + j) + (lane & 15);
        if (n >= a.d_out) continue;
        float bl[BSQ_MAX_LORA_RANK];
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) bl[q] = (q < a.rank) ? bf16_to_f32(a.B[n * a.rank + q]) : 0.0f;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t m = m0 + 16 * i + 4 * (lane >> 4) + r;
                if (m >= a.M) continue;
                float v = acc[i][j][r];
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
}

template <int D, int S>
hipError_t launch_gemm_t(const GemmArgs &a, hipStream_t st)
{
    const int64_t nrg = (a.d_out + 63) / 64;
    const size_t shm = size_t((a.words + 3) & ~int64_t(3)) * 4 + ((D == 8) ? size_t(S) * 256 * 8 * 4 : 0);
    const dim3 block = dim3(256);
    if (a.M <= 16) {
        hipLaunchKernelGGL((gemm_kernel<D, S, 1, 1>), dim3(unsigned(nrg), unsigned((a.M + 15) / 16)), block, shm, st, a);
    } else if (a.M <= 64) {
        hipLaunchKernelGGL((gemm_kernel<D, S, 4, 1>), dim3(unsigned(nrg), unsigned((a.M + 63) / 64)), block, shm, st, a);
    } else if (a.M <= 128) {
        hipLaunchKernelGGL((gemm_kernel<D, S, 4, 2>), dim3(unsigned(nrg), unsigned((a.M + 127) / 128)), block, shm, st, a);
    } else {
        hipLaunchKernelGGL((gemm_kernel<D, S, 4, 4>), dim3(unsigned(nrg), unsigned((a.M + 255) / 256)), block, shm, st, a);
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
