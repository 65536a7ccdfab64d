// Decoder tables: each stage decoder D_s evaluated on all 2^b spherical codes
// (Section III-C: q_j = +-1/sqrt(b); Section IV-D: identity, linear and the
// compact symmetric decoder with one hidden ReLU layer, without or with one
// residual block on that layer). The fp32 table is
// filled with the same fmaf chains, in the same element order, as the
// definition of the encoder, so that encode and decode are exact; the bf16
// table (round to nearest even) feeds the GEMV's products, the fp16 table
// (round to nearest even) the GEMM's decode. For the symmetric decoder at
// d = 16 the hidden pre-activation is also tabulated per code byte (two
// halves whose entries add up to it), the form the d = 16 GEMV evaluates.
#include "bsq_internal.h"

namespace bsq {
namespace {

struct TableArgs {
    const float *W1[BSQ_MAX_STAGES];
    const float *b1[BSQ_MAX_STAGES];
    const float *W2[BSQ_MAX_STAGES];
    const float *b2[BSQ_MAX_STAGES];
    const float *R[BSQ_MAX_STAGES];   // residual block [h][h], [h] (res1 only)
    const float *c[BSQ_MAX_STAGES];
    float *t32[BSQ_MAX_STAGES];
    uint16_t *t16[BSQ_MAX_STAGES];
    uint16_t *th[BSQ_MAX_STAGES];
    float cscale;  // (float)(1 / sqrt(b)), rounded once from double
    int kind;
    int hidden;
};

// D outputs per code, B code bits (B = D unless the codec has a linear encoder)
template <int D, int B>
__global__ __launch_bounds__(256) void codec_table_kernel(TableArgs a)
{
    const int s = blockIdx.y;
    const uint32_t code = blockIdx.x * blockDim.x + threadIdx.x;
    if (code >= (1u << B)) return;

    float q[B];
#pragma unroll
    for (int j = 0; j < B; ++j) q[j] = ((code >> j) & 1u) ? a.cscale : -a.cscale;

    float y[D];
    if (a.kind == BSQ_DEC_IDENTITY) {  // (B = D)
#pragma unroll
        for (int j = 0; j < D; ++j) y[j] = q[j % B];
    } else if (a.kind == BSQ_DEC_LINEAR) {
        const float *M = a.W1[s];
        const float *beta = a.b1[s];
#pragma unroll
        for (int m = 0; m < D; ++m) {
            float acc = beta[m];
#pragma unroll
            for (int j = 0; j < B; ++j) acc = __builtin_fmaf(M[m * B + j], q[j], acc);
            y[m] = acc;
        }
    } else {
        const float *W1 = a.W1[s], *b1 = a.b1[s], *W2 = a.W2[s], *b2 = a.b2[s];
        const int h = a.hidden;
        float act[BSQ_MAX_HIDDEN];
        for (int k = 0; k < h; ++k) {
            float acc = b1[k];
#pragma unroll
            for (int j = 0; j < B; ++j) acc = __builtin_fmaf(W1[k * B + j], q[j], acc);
            act[k] = (acc > 0.0f) ? acc : 0.0f;
        }
        if (a.kind == BSQ_DEC_MLP_RES1) {
            // a' = a + relu(c + R a): every t_k from the unmodified a, then the adds
            const float *R = a.R[s], *c = a.c[s];
            float t[BSQ_MAX_HIDDEN];
            for (int k = 0; k < h; ++k) {
                float acc = c[k];
                for (int l = 0; l < h; ++l) acc = __builtin_fmaf(R[k * h + l], act[l], acc);
                t[k] = (acc > 0.0f) ? acc : 0.0f;
            }
            for (int k = 0; k < h; ++k) act[k] = act[k] + t[k];
        }
#pragma unroll
        for (int m = 0; m < D; ++m) {
            float acc = b2[m];
            for (int k = 0; k < h; ++k) acc = __builtin_fmaf(W2[m * h + k], act[k], acc);
            y[m] = acc;
        }
    }
    float *o32 = a.t32[s] + size_t(code) * D;
    uint16_t *o16 = a.t16[s] + size_t(code) * D;
    uint16_t *oh = a.th[s] + size_t(code) * D;
#pragma unroll
    for (int m = 0; m < D; ++m) {
        o32[m] = y[m];
        o16[m] = f32_to_bf16(y[m]);
        oh[m] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(y[m]));
    }
}

struct SplitArgs {
    const float *W1[BSQ_MAX_STAGES];
    const float *b1[BSQ_MAX_STAGES];
    const float *W2[BSQ_MAX_STAGES];
    const float *b2[BSQ_MAX_STAGES];
    uint16_t *split[BSQ_MAX_STAGES];  // fp16 [2][256][h]
    float *w2[BSQ_MAX_STAGES];        // fp32 [16][h]
    float *b2c[BSQ_MAX_STAGES];       // fp32 [16]
    float cscale;
    int hidden;
};

// One block per stage, one thread per byte v: half 0 of the hidden
// pre-activation is the fmaf chain b1_k + sum_{j<8} W1[k][j] q_j(v), half 1
// the chain 0 + sum_{j<8} W1[k][8 + j] q_j(v) (q_j(v) = +c if bit j of v is
// set, else -c), both rounded to fp16 (nearest even). Stored as
// [half][k / 8][v][k % 8]: the 16-byte groups of eight hidden units of all
// bytes v are contiguous, so that a lookup's 16-byte reads spread over every
// LDS bank.
__global__ __launch_bounds__(256) void codec_split_kernel(SplitArgs a)
{
    const int s = blockIdx.x;
    const uint32_t v = threadIdx.x;
    const int h = a.hidden;
    const float *W1 = a.W1[s];
    float q[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = ((v >> j) & 1u) ? a.cscale : -a.cscale;
    for (int half = 0; half < 2; ++half) {
        for (int k = 0; k < h; ++k) {
            float acc = half ? 0.0f : a.b1[s][k];
#pragma unroll
            for (int j = 0; j < 8; ++j) acc = __builtin_fmaf(W1[k * 16 + 8 * half + j], q[j], acc);
            a.split[s][((size_t(half) * ((h + 7) / 8) + k / 8) * 256 + v) * 8 + k % 8] =
                __builtin_bit_cast(uint16_t, static_cast<_Float16>(acc));
        }
    }
    for (int e = int(v); e < 16 * h; e += 256) a.w2[s][e] = a.W2[s][e];
    if (v < 16) a.b2c[s][v] = a.b2[s][v];
}

}  // namespace

hipError_t launch_codec_tables(const bsq_config &cfg, const bsq_decoder *dec, void *codec, hipStream_t st)
{
    TableArgs a{};
    char *base = static_cast<char *>(codec);
    for (int s = 0; s < cfg.stages; ++s) {
        a.W1[s] = dec[s].W1;
        a.b1[s] = dec[s].b1;
        a.W2[s] = dec[s].W2;
        a.b2[s] = dec[s].b2;
        a.R[s] = dec[s].R;
        a.c[s] = dec[s].c;
        a.t32[s] = reinterpret_cast<float *>(base + codec_tab32_offset(cfg, s));
        a.t16[s] = reinterpret_cast<uint16_t *>(base + codec_tab16_offset(cfg, s));
        a.th[s] = reinterpret_cast<uint16_t *>(base + codec_tabh_offset(cfg, s));
    }
    a.cscale = float(1.0 / __builtin_sqrt(double(cfg.b)));
    a.kind = cfg.dec_kind;
    a.hidden = cfg.hidden;
    const uint32_t ncodes = 1u << cfg.b;
    dim3 grid((ncodes + 255) / 256, cfg.stages);
    if (cfg.d == 8 && cfg.b == 8)
        hipLaunchKernelGGL((codec_table_kernel<8, 8>), grid, dim3(256), 0, st, a);
    else if (cfg.d == 16 && cfg.b == 16)
        hipLaunchKernelGGL((codec_table_kernel<16, 16>), grid, dim3(256), 0, st, a);
    else if (cfg.d == 8)
        hipLaunchKernelGGL((codec_table_kernel<8, 16>), grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL((codec_table_kernel<16, 8>), grid, dim3(256), 0, st, a);
    if (codec_has_split(cfg)) {
        SplitArgs sa{};
        for (int s = 0; s < cfg.stages; ++s) {
            sa.W1[s] = dec[s].W1;
            sa.b1[s] = dec[s].b1;
            sa.W2[s] = dec[s].W2;
            sa.b2[s] = dec[s].b2;
            sa.split[s] = reinterpret_cast<uint16_t *>(base + codec_split_offset(cfg, s));
            sa.w2[s] = reinterpret_cast<float *>(base + codec_w2_offset(cfg, s));
            sa.b2c[s] = reinterpret_cast<float *>(base + codec_b2_offset(cfg, s));
        }
        sa.cscale = a.cscale;
        sa.hidden = cfg.hidden;
        hipLaunchKernelGGL(codec_split_kernel, dim3(unsigned(cfg.stages)), dim3(256), 0, st, sa);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // the encoders travel with the codec, which is all bsq_encode receives
    for (int s = 0; s < cfg.stages && cfg.encoder == BSQ_ENC_LINEAR; ++s) {
        e = hipMemcpyAsync(base + codec_enc_offset(cfg, s), dec[s].E, size_t(cfg.b) * cfg.d * 4,
                           hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace bsq
