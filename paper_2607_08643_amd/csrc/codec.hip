// Decoder tables: each stage decoder D_s evaluated on all 2^b spherical codes
// (Section III-C: q_j = +-1/sqrt(b); Section IV-D: identity, linear and the
// compact symmetric decoder with one hidden ReLU layer). The fp32 table is
// filled with the same fmaf chains, in the same element order, as the
// definition of the encoder, so that encode and decode are exact; the bf16
// table (round to nearest even) feeds the GEMV's products, the fp16 table
// (round to nearest even) the GEMM's decode.
#include "bsq_internal.h"

namespace bsq {
namespace {

struct TableArgs {
    const float *W1[BSQ_MAX_STAGES];
    const float *b1[BSQ_MAX_STAGES];
    const float *W2[BSQ_MAX_STAGES];
    const float *b2[BSQ_MAX_STAGES];
    float *t32[BSQ_MAX_STAGES];
    uint16_t *t16[BSQ_MAX_STAGES];
    uint16_t *th[BSQ_MAX_STAGES];
    float cscale;  // (float)(1 / sqrt(b)), rounded once from double
    int kind;
    int hidden;
};

template <int D>
__global__ __launch_bounds__(256) void codec_table_kernel(TableArgs a)
{
    const int s = blockIdx.y;
    const uint32_t code = blockIdx.x * blockDim.x + threadIdx.x;
    if (code >= (1u << D)) return;

    float q[D];
#pragma unroll
    for (int j = 0; j < D; ++j) q[j] = ((code >> j) & 1u) ? a.cscale : -a.cscale;

    float y[D];
    if (a.kind == BSQ_DEC_IDENTITY) {
#pragma unroll
        for (int j = 0; j < D; ++j) y[j] = q[j];
    } else if (a.kind == BSQ_DEC_LINEAR) {
        const float *M = a.W1[s];
        const float *beta = a.b1[s];
#pragma unroll
        for (int m = 0; m < D; ++m) {
            float acc = beta[m];
#pragma unroll
            for (int j = 0; j < D; ++j) acc = __builtin_fmaf(M[m * D + j], q[j], acc);
            y[m] = acc;
        }
    } else {
        const float *W1 = a.W1[s], *b1 = a.b1[s], *W2 = a.W2[s], *b2 = a.b2[s];
        const int h = a.hidden;
        float act[BSQ_MAX_HIDDEN];
        for (int k = 0; k < h; ++k) {
            float acc = b1[k];
#pragma unroll
            for (int j = 0; j < D; ++j) acc = __builtin_fmaf(W1[k * D + j], q[j], acc);
            act[k] = (acc > 0.0f) ? acc : 0.0f;
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
        a.t32[s] = reinterpret_cast<float *>(base + codec_tab32_offset(cfg, s));
        a.t16[s] = reinterpret_cast<uint16_t *>(base + codec_tab16_offset(cfg, s));
        a.th[s] = reinterpret_cast<uint16_t *>(base + codec_tabh_offset(cfg, s));
    }
    a.cscale = float(1.0 / __builtin_sqrt(double(cfg.b)));
    a.kind = cfg.dec_kind;
    a.hidden = cfg.hidden;
    const uint32_t ncodes = 1u << cfg.b;
    dim3 grid((ncodes + 255) / 256, cfg.stages);
    if (cfg.d == 8)
        hipLaunchKernelGGL(codec_table_kernel<8>, grid, dim3(256), 0, st, a);
    else
        hipLaunchKernelGGL(codec_table_kernel<16>, grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace bsq
