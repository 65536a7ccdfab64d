// Internal declarations of libbsq: codec buffer layout, device helpers and
// the host-side launchers of every kernel. Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/bsq.h"

namespace bsq {

// ---------------------------------------------------------------------------
// Codec buffer: for each stage an fp32 table [2^b][d] (exact decoder values),
// then for each stage a bf16 table [2^b][d] (the same values rounded to
// nearest even, consumed by the GEMV's bf16 products), then for each stage an
// fp16 table [2^b][d] (rounded to nearest even, consumed by the GEMM's decode
// through mixed-precision fma).
//
// The table has 2^b entries of d values (b = d with the identity encoder).
// The symmetric decoder at d = b = 16 also gets, per stage, its hidden
// pre-activation split by code byte: fp16 [2][h/8][256][8], half 0 holding
// b1 + W1[:, 0:8] q(v) and half 1 W1[:, 8:16] q(v) for every byte v (so the
// pre-activation of a code is the sum of one entry of each half; each entry
// is stored as h/8 groups of eight units, 16 bytes each), followed by fp32
// copies of W2 [d][h] and b2 [d]. The GEMV folds W2 and b2 into the
// activations and evaluates the decoder from these halves.
// ---------------------------------------------------------------------------
inline size_t codec_entries(const bsq_config &c) { return (size_t(1) << c.b) * size_t(c.d); }
inline size_t codec_tab32_offset(const bsq_config &c, int s) { return size_t(s) * codec_entries(c) * 4; }
inline size_t codec_tab16_offset(const bsq_config &c, int s)
{
    return size_t(c.stages) * codec_entries(c) * 4 + size_t(s) * codec_entries(c) * 2;
}
inline size_t codec_tabh_offset(const bsq_config &c, int s)
{
    return size_t(c.stages) * codec_entries(c) * 6 + size_t(s) * codec_entries(c) * 2;
}
// (the residual-block decoder is not split: its block mixes the hidden units)
inline bool codec_has_split(const bsq_config &c) { return c.dec_kind == BSQ_DEC_MLP && c.d == 16 && c.b == 16; }
// one stage's split tables and decoder copies
inline size_t codec_split_stage_bytes(const bsq_config &c)
{
    return codec_has_split(c) ? size_t(2) * 256 * c.hidden * 2 + size_t(c.d) * c.hidden * 4 + size_t(c.d) * 4 : 0;
}
inline size_t codec_split_offset(const bsq_config &c, int s)
{
    return size_t(c.stages) * codec_entries(c) * 8 + size_t(s) * codec_split_stage_bytes(c);
}
inline size_t codec_w2_offset(const bsq_config &c, int s)
{
    return codec_split_offset(c, s) + size_t(2) * 256 * c.hidden * 2;
}
inline size_t codec_b2_offset(const bsq_config &c, int s) { return codec_w2_offset(c, s) + size_t(c.d) * c.hidden * 4; }
// then, with a linear encoder, a copy of each stage's E [b][d] (fp32)
inline size_t codec_enc_offset(const bsq_config &c, int s)
{
    return size_t(c.stages) * codec_entries(c) * 8 + size_t(c.stages) * codec_split_stage_bytes(c) +
           size_t(s) * c.b * c.d * 4;
}
inline size_t codec_total_bytes(const bsq_config &c)
{
    return codec_enc_offset(c, c.encoder == BSQ_ENC_LINEAR ? c.stages : 0);
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// ---------------------------------------------------------------------------
// Tiled plane layout of the code and gain planes: 64-row x 16-chunk tiles,
// [n_mats][ceil(d_out / 64)][pitch / 16][64][16]. A wave that owns 64 rows
// and one 16-chunk block reads one contiguous tile with one 16-byte load per
// lane per code plane (d = 8); a 64-row x 128-input weight tile of the GEMM
// (d = 8) is exactly one tile.
// ---------------------------------------------------------------------------
__host__ __device__ inline int64_t tile_index(int64_t row, int64_t chunk, int64_t pitch)
{
    return ((((row >> 6) * (pitch >> 4)) + (chunk >> 4)) << 10) + ((row & 63) << 4) + (chunk & 15);
}
__host__ __device__ inline int64_t plane_elems(int64_t d_out, int64_t pitch) { return ((d_out + 63) >> 6) * 64 * pitch; }

// ---------------------------------------------------------------------------
// Device helpers.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// fp32 -> bf16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u) return uint16_t((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// Two fp32 values rounded to bf16 (nearest even, as f32_to_bf16 for every
// non-NaN input) in one v_cvt_pk_bf16_f32; lo in the low half.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi)
{
    typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
    typedef float f32x2_v __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_v{lo, hi}, bf16x2_v));
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h)
{
    _Float16 v;
    __builtin_memcpy(&v, &h, 2);
    return float(v);
}

// Gain storage rule: fp16 round to nearest even (hardware conversion in the
// default rounding mode), finite overflow saturated to +-65504.
__device__ __forceinline__ uint16_t gain_to_f16(float a)
{
    _Float16 h = _Float16(a);
    uint16_t u;
    __builtin_memcpy(&u, &h, 2);
    if ((u & 0x7fffu) == 0x7c00u) u = uint16_t((u & 0x8000u) | 0x7bffu);
    return u;
}

// ---------------------------------------------------------------------------
// Protected payload formats (bsq_prot_format): one stored byte per protected
// element; its value times the slice's fp32 scale is the weight, and the
// scale is the slice's largest magnitude over payload_max.
// ---------------------------------------------------------------------------
__host__ __device__ inline float payload_max(int fmt)
{
    return fmt == BSQ_PROT_E4M3 ? 448.0f : (fmt == BSQ_PROT_E5M2 ? 57344.0f : 127.0f);
}

// The value of byte SEL of a word of stored bytes: int8 two's complement, or
// the OCP FP8 fields (E4M3: bias 7, S.1111.111 NaN; E5M2: bias 15, exponent
// 31 infinity or NaN; exponent 0 subnormal in both), read by gfx950's
// conversion instructions, which implement exactly these formats (every one
// of the 256 bytes of both formats is checked against their definitions).
template <int FMT, int SEL>
__device__ __forceinline__ float payload_byte(uint32_t word)
{
    if constexpr (FMT == BSQ_PROT_E4M3) return __builtin_amdgcn_cvt_f32_fp8(int(word), SEL);
    else if constexpr (FMT == BSQ_PROT_E5M2) return __builtin_amdgcn_cvt_f32_bf8(int(word), SEL);
    else return float(int8_t(uint8_t(word >> (8 * SEL))));
}

// The value of the stored byte in the low 8 bits of q.
template <int FMT>
__device__ __forceinline__ float payload_value(uint32_t q)
{
    return payload_byte<FMT, 0>(q);
}

// The same with the format known at run time only (one uniform dispatch).
__device__ __forceinline__ float payload_to_f32(uint32_t q, int fmt)
{
    if (fmt == BSQ_PROT_E4M3) return payload_value<BSQ_PROT_E4M3>(q);
    if (fmt == BSQ_PROT_E5M2) return payload_value<BSQ_PROT_E5M2>(q);
    return payload_value<BSQ_PROT_INT8>(q);
}

// The stored byte of v (a weight over its slice's scale). int8: round half
// to even, clamped to +-127. FP8: the nearest finite value, ties to the even
// code, sign kept, magnitudes from the largest finite value up stored as it.
// Below the smallest normal 2^emin the steps are 2^(emin - mb); in the
// binade [2^e, 2^(e+1)) they are 2^(e - mb), so the scaled magnitude is
// rounded once to an integer n (exact power-of-two scalings, round to nearest
// even) and n = 2^(mb+1) carries into the next exponent by itself.
__device__ __forceinline__ uint32_t payload_from_f32(float v, int fmt)
{
    if (fmt == BSQ_PROT_INT8) {
        float t = __builtin_rintf(v);
        t = (t > 127.0f) ? 127.0f : t;
        t = (t < -127.0f) ? -127.0f : t;
        return uint32_t(uint8_t(int8_t(t)));
    }
    const bool e4 = fmt == BSQ_PROT_E4M3;
    const int mb = e4 ? 3 : 2, bias = e4 ? 7 : 15, emin = 1 - bias;
    const uint32_t sign = (__float_as_uint(v) >> 24) & 0x80u;
    const float a = __builtin_fabsf(v);
    if (a >= payload_max(fmt)) return sign | (e4 ? 0x7eu : 0x7bu);
    if (a < __builtin_ldexpf(1.0f, emin)) return sign | uint32_t(__builtin_rintf(__builtin_ldexpf(a, mb - emin)));
    const int e = int((__float_as_uint(a) >> 23) & 0xffu) - 127;
    const uint32_t n = uint32_t(__builtin_rintf(__builtin_ldexpf(a, mb - e)));
    return sign | ((uint32_t(e + bias) << mb) + (n - (1u << mb)));
}

// ---------------------------------------------------------------------------
// Launchers (defined in the .hip files; all asynchronous on `st`).
// ---------------------------------------------------------------------------
hipError_t launch_codec_tables(const bsq_config &cfg, const bsq_decoder *dec, void *codec, hipStream_t st);

struct EncodeWs {
    double *keys;       // [n_mats][n], n = d_in (column axis) or d_out (row axis)
    float *absmax;      // [n_mats][n]
    int32_t *colmap;    // [n_mats][n]: protected column -> its position p
    uint32_t *bits;     // row axis: the row selection's bitmap (unused)
};

struct SelectWs {       // coupled MLP selection, all [d_ffn]
    double *sg, *su, *sd, *keys;
    float *absmax, *scale;
    int32_t *colmap;
    uint32_t *bits;
};

// protected payload row length: k protected columns padded to a multiple of 16
// (zero bytes), so that one row is read with 16-byte loads
__host__ __device__ inline int64_t q8_pitch(int64_t k) { return (k + 15) & ~int64_t(15); }

// 32-bit words of a layer's protected-column bitmap: one bit per padded column
__host__ __device__ inline int64_t prot_words(int64_t pitch, int d) { return pitch * d / 32; }
size_t encode_ws_layout(const bsq_config &cfg, int64_t n_mats, int64_t d_out, int64_t d_in, char *base,
                        EncodeWs *ws);
size_t select_ws_layout(int64_t d_ffn, char *base, SelectWs *ws);
// `given`: a caller's protected set (device int32 [n_mats][k]), or nullptr to select one
hipError_t launch_encode(const bsq_config &cfg, const void *codec, const void *W, int w_dtype,
                         int64_t n_mats, int64_t d_out, int64_t d_in, const float *g, const int32_t *given,
                         const bsq_layer &out, int32_t *err, const EncodeWs &ws, hipStream_t st);
hipError_t launch_coupled_select(const void *Wg, const void *Wu, const void *Wd, int w_dtype, int64_t d_model,
                                 int64_t d_ffn, const float *gg, const float *gu, const float *gd, int64_t k,
                                 int32_t *idx, double *scores, int32_t *err, const SelectWs &ws, hipStream_t st);
// protected output rows of the products (run after the streaming kernels, same stream)
// (`fmt`: the payload's bsq_prot_format)
hipError_t launch_decode_rows(const bsq_layer &layer, int fmt, void *w_hat, int out_dtype, hipStream_t st);
hipError_t launch_gemv_rows(int n, const bsq_layer *layers, int fmt, const bsq_lora *loras, const void *x,
                            int x_dtype, void *const *y, int y_dtype, hipStream_t st);
hipError_t launch_gemm_rows(const bsq_layer &layer, int fmt, const bsq_lora *lora, const void *X, int64_t M,
                            int64_t ldx, void *Y, int y_dtype, int64_t ldy, const float *T, hipStream_t st);
// X A^T (fp32 [Mp][BSQ_MAX_LORA_RANK]) as left in a GEMM workspace by launch_gemm
const float *gemm_lora_t(const void *ws);

hipError_t launch_decode(const bsq_config &cfg, const void *codec, const bsq_layer &layer,
                         void *w_hat, int out_dtype, hipStream_t st);
hipError_t launch_decode_stage(const bsq_config &cfg, const void *codec, const bsq_layer &layer, int stage,
                               int accumulate, void *w_hat, hipStream_t st);

size_t gemv_ws_bytes(const bsq_config &cfg, int64_t n, int64_t max_d_out, int64_t d_in);
// The device address of the current device's bsq_gemv_noalloc scratch array
// (BSQ_GEMV_NOALLOC_SCRATCH_BYTES, 256-byte aligned); on the first call on a
// device, or with `clear`, a zero-fill of the array is launched on `st`.
hipError_t gemv_scratch(bool clear, void **ptr, hipStream_t st);
// `scratch_layout`: ws is bsq_gemv_noalloc's shared scratch array, whose
// layout does not depend on the call's shape (see make_args)
hipError_t launch_gemv_prep(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                            const bsq_lora *loras, const void *x, int x_dtype, void *ws, bool scratch_layout,
                            hipStream_t st);
hipError_t launch_gemv_run(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                           const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype,
                           void *ws, bool scratch_layout, int32_t *err, hipStream_t st);
// whether a group's workspace fits the scratch array in its scratch layout
bool gemv_scratch_fits(const bsq_config &cfg, int64_t n, int64_t max_d_out, int64_t d_in);

size_t gemm_ws_bytes(const bsq_config &cfg, int64_t d_out, int64_t d_in, int64_t M);
hipError_t launch_gemm(const bsq_config &cfg, const void *codec, const bsq_layer &layer,
                       const bsq_lora *lora, const void *X, int64_t M, int64_t ldx, void *Y,
                       int y_dtype, int64_t ldy, void *ws, int32_t *err, hipStream_t st);

// Codec training (train.hip): parameters of one stage codec, floats per chunk
// record, workspace bytes for a batch of n chunks, and the two launches.
int64_t train_param_count(const bsq_config &cfg);
int64_t train_record_floats(const bsq_config &cfg);
size_t train_ws_bytes(const bsq_config &cfg, int64_t n);
hipError_t launch_train_grad(const bsq_config &cfg, const bsq_train_hparams &hp, const void *x, int x_dtype,
                             int64_t n_total, const int64_t *idx, int64_t n, const float *theta, float *grad,
                             float *loss, int32_t *err, void *ws, hipStream_t st);
hipError_t launch_train_adam(const bsq_config &cfg, const bsq_train_hparams &hp, int step, float *theta,
                             const float *grad, float *m, float *v, hipStream_t st);

// Polls a finishing workgroup makes for another workgroup's partial result
// before it gives up (reports BSQ_DEVERR_TIMEOUT and poisons the workspace).
// Workgroups run in dispatch order, so the wait is never expected to give
// up; bsq_debug_set_wait_limit lowers the bound so that tests can force it.
int wait_limit();

}  // namespace bsq
