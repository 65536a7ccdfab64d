// C ABI of libbsq.so (include/bsq.h): host-side validation of every argument
// before anything is launched, then dispatch to the kernels.
#include <cmath>

#include "bsq_internal.h"

using namespace bsq;

namespace {

bool aligned(const void *p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// protected slices of a d_out x d_in matrix on the config's axis
int64_t k_of(const bsq_config &c, int64_t d_out, int64_t d_in)
{
    if (c.protect_num == 0) return 0;
    const int64_t n = (c.protect_axis == 1) ? d_out : d_in;
    return (n * c.protect_num + c.protect_den - 1) / c.protect_den;
}

bool row_axis(const bsq_config &c) { return c.protect_axis == 1 && c.protect_num > 0; }

// The configuration and layer the streaming kernels see: with protected rows
// they code every row with no column masked (the protected rows' code 0 and
// gain +0 contribute nothing), and the rows kernels write the protected rows.
bsq_config coded_cfg(const bsq_config &c)
{
    bsq_config r = c;
    if (row_axis(c)) r.protect_num = 0;
    return r;
}

bsq_layer coded_layer(const bsq_config &c, const bsq_layer &L)
{
    bsq_layer r = L;
    if (row_axis(c)) {
        r.k = 0;
        r.prot_idx = nullptr;
        r.prot_q8 = nullptr;
        r.prot_scale = nullptr;
        r.prot_bits = nullptr;
    }
    return r;
}

int64_t pitch_of(const bsq_config &c, int64_t d_in)
{
    const int64_t C = d_in / c.d;
    return (C + BSQ_PITCH_ALIGN - 1) / BSQ_PITCH_ALIGN * BSQ_PITCH_ALIGN;
}

bsq_status check_cfg(const bsq_config *c)
{
    if (!c) return BSQ_ERR_ARG;
    if (c->d < 1 || c->d > 16 || c->b < 1 || c->b > 16) return BSQ_ERR_ARG;
    if (c->stages < 1 || c->stages > BSQ_MAX_STAGES) return BSQ_ERR_ARG;
    if (c->dec_kind < BSQ_DEC_IDENTITY || c->dec_kind > BSQ_DEC_MLP_RES1) return BSQ_ERR_ARG;
    if ((c->dec_kind == BSQ_DEC_MLP || c->dec_kind == BSQ_DEC_MLP_RES1) &&
        (c->hidden < 1 || c->hidden > BSQ_MAX_HIDDEN))
        return BSQ_ERR_ARG;
    if (c->protect_format < BSQ_PROT_INT8 || c->protect_format > BSQ_PROT_E5M2) return BSQ_ERR_ARG;
    if (c->protect_num < 0 || c->protect_den < 1 || c->protect_num > c->protect_den) return BSQ_ERR_ARG;
    if (c->protect_axis != 0 && c->protect_axis != 1) return BSQ_ERR_ARG;
    if (c->encoder != BSQ_ENC_IDENTITY && c->encoder != BSQ_ENC_LINEAR) return BSQ_ERR_ARG;
    if (c->d != 8 && c->d != 16) return BSQ_ERR_UNSUPPORTED;
    if (c->b != 8 && c->b != 16) return BSQ_ERR_UNSUPPORTED;
    // b != d needs an encoder R^d -> R^b; the identity decoder needs b = d
    if (c->b != c->d && (c->encoder == BSQ_ENC_IDENTITY || c->dec_kind == BSQ_DEC_IDENTITY)) return BSQ_ERR_ARG;
    return BSQ_OK;
}

bsq_status check_shape(const bsq_config &c, int64_t d_out, int64_t d_in)
{
    if (d_out < 0 || d_in < 1) return BSQ_ERR_SHAPE;
    if (d_in % c.d != 0) return BSQ_ERR_SHAPE;
    if (d_in > (int64_t(1) << 18) || d_out > (int64_t(1) << 31)) return BSQ_ERR_UNSUPPORTED;
    return BSQ_OK;
}

bsq_status check_layer(const bsq_config &c, const bsq_layer *L, bool need_planes, bool need_bits)
{
    if (!L) return BSQ_ERR_ARG;
    bsq_status s = check_shape(c, L->d_out, L->d_in);
    if (s != BSQ_OK) return s;
    if (L->n_mats < 1) return BSQ_ERR_ARG;
    if (L->pitch != pitch_of(c, L->d_in)) return BSQ_ERR_ARG;
    if (L->k != k_of(c, L->d_out, L->d_in)) return BSQ_ERR_ARG;
    if (need_planes && L->d_out > 0) {
        for (int i = 0; i < c.stages; ++i) {
            if (!L->codes[i] || !L->gains[i]) return BSQ_ERR_ARG;
            if (!aligned(L->codes[i], 16) || !aligned(L->gains[i], 16)) return BSQ_ERR_ALIGN;
        }
    }
    if (row_axis(c)) {
        // protected rows: indices, scales and the [k][q8_pitch(d_in)] payload
        if (L->k > 0 && (!L->prot_idx || !L->prot_scale || !L->prot_q8)) return BSQ_ERR_ARG;
        if (L->k > 0 && (!aligned(L->prot_idx, 4) || !aligned(L->prot_scale, 4) || !aligned(L->prot_q8, 16)))
            return BSQ_ERR_ALIGN;
        if (L->k > 0 && L->d_in > (int64_t(1) << 18)) return BSQ_ERR_UNSUPPORTED;
        return BSQ_OK;
    }
    if (L->k > 0 && (!L->prot_idx || !L->prot_scale)) return BSQ_ERR_ARG;
    if (L->k > 0 && L->d_out > 0 && !L->prot_q8) return BSQ_ERR_ARG;
    if (L->k > 0 && !aligned(L->prot_idx, 4)) return BSQ_ERR_ALIGN;
    if (L->k > 0 && L->d_out > 0 && !aligned(L->prot_q8, 16)) return BSQ_ERR_ALIGN;
    if (L->k > 0 && !aligned(L->prot_scale, 4)) return BSQ_ERR_ALIGN;
    if (need_bits && L->k > 0 && !L->prot_bits) return BSQ_ERR_ARG;
    if (need_bits && L->k > 0 && !aligned(L->prot_bits, 16)) return BSQ_ERR_ALIGN;
    return BSQ_OK;
}

bsq_status check_lora(const bsq_lora *l)
{
    if (!l || l->rank == 0) return BSQ_OK;
    if (l->rank < 0 || l->rank > BSQ_MAX_LORA_RANK) return BSQ_ERR_ARG;
    if (!l->A || !l->B) return BSQ_ERR_ARG;
    if (!aligned(l->A, 2) || !aligned(l->B, 2)) return BSQ_ERR_ALIGN;
    return BSQ_OK;
}

bsq_status from_hip(hipError_t e) { return e == hipSuccess ? BSQ_OK : BSQ_ERR_DEVICE; }

// polls before a finishing workgroup's wait gives up: about a second of
// s_sleep polling by default (never expected to be reached, since workgroups
// run in dispatch order); bsq_debug_set_wait_limit changes it
constexpr int32_t DEFAULT_WAIT_LIMIT = 1 << 22;
int32_t g_wait_limit = DEFAULT_WAIT_LIMIT;

}  // namespace

namespace bsq {
int wait_limit() { return __atomic_load_n(&g_wait_limit, __ATOMIC_RELAXED); }
}  // namespace bsq

extern "C" {

int32_t bsq_version(void) { return BSQ_ABI_VERSION; }

int32_t bsq_debug_set_wait_limit(int32_t polls)
{
    const int32_t prev = __atomic_load_n(&g_wait_limit, __ATOMIC_RELAXED);
    __atomic_store_n(&g_wait_limit, polls < 0 ? DEFAULT_WAIT_LIMIT : polls, __ATOMIC_RELAXED);
    return prev;
}

const char *bsq_status_str(int32_t s)
{
    switch (s) {
    case BSQ_OK: return "ok";
    case BSQ_ERR_ARG: return "invalid argument";
    case BSQ_ERR_SHAPE: return "invalid shape";
    case BSQ_ERR_DTYPE: return "unsupported dtype";
    case BSQ_ERR_ALIGN: return "misaligned buffer";
    case BSQ_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case BSQ_ERR_NONFINITE: return "non-finite input";
    case BSQ_ERR_DEVICE: return "device error";
    case BSQ_ERR_UNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
    }
}

bsq_status bsq_config_check(const bsq_config *cfg) { return check_cfg(cfg); }

bsq_status bsq_layer_sizes(const bsq_config *cfg, int64_t d_out, int64_t d_in, int32_t lora_rank, bsq_sizes *out)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!out) return BSQ_ERR_ARG;
    if ((s = check_shape(*cfg, d_out, d_in)) != BSQ_OK) return s;
    if (lora_rank < 0 || lora_rank > BSQ_MAX_LORA_RANK) return BSQ_ERR_ARG;
    const bsq_config &c = *cfg;
    const int64_t C = d_in / c.d, k = k_of(c, d_out, d_in), P = pitch_of(c, d_in);
    const bool rows = row_axis(c);
    // protected rows are not BSQ-coded: their all-zero plane rows are layout,
    // not payload
    const int64_t coded_rows = rows ? d_out - k : d_out;
    const int64_t code_bytes = (c.b <= 8) ? 1 : 2;
    out->pitch = P;
    out->k = k;
    out->chunks = d_out * C;
    out->code_plane_bytes = plane_elems(d_out, P) * code_bytes;
    out->gain_plane_bytes = plane_elems(d_out, P) * 2;
    out->idx_bytes = k * 4;
    out->q8_bytes = rows ? k * q8_pitch(d_in) : d_out * q8_pitch(k);
    out->scale_bytes = k * 4;
    out->bits_bytes = (k > 0 && !rows) ? prot_words(P, c.d) * 4 : 0;
    int64_t dec_params = 0;
    if (c.dec_kind == BSQ_DEC_MLP || c.dec_kind == BSQ_DEC_MLP_RES1)
        dec_params = int64_t(c.hidden) * c.b + c.hidden + int64_t(c.d) * c.hidden + c.d;
    else if (c.dec_kind == BSQ_DEC_LINEAR)
        dec_params = int64_t(c.d) * c.b + c.d;
    if (c.dec_kind == BSQ_DEC_MLP_RES1) dec_params += int64_t(c.hidden) * c.hidden + c.hidden;
    if (c.encoder == BSQ_ENC_LINEAR) dec_params += int64_t(c.b) * c.d;
    out->S_code = double(c.stages) * double(coded_rows) * double(C) * double(c.b) / 8.0;
    out->S_dec = double(c.stages) * double(dec_params) * 4.0;
    out->S_8bit = rows ? double(k) * double(d_in) : double(d_out) * double(k);
    out->S_LoRA = 2.0 * double(lora_rank) * double(d_in + d_out);
    out->S_meta = double(c.stages) * double(coded_rows) * double(C) * 2.0 + 8.0 * double(k);
    out->S_tot = out->S_code + out->S_dec + out->S_8bit + out->S_LoRA + out->S_meta;
    out->bpw_nominal = double(c.stages) * double(c.b) / double(c.d);
    out->bpw_real = (d_out > 0) ? 8.0 * out->S_tot / (double(d_out) * double(d_in)) : 0.0;
    return BSQ_OK;
}

bsq_status bsq_workspace_bytes(const bsq_config *cfg, int32_t op, int64_t n_mats, int64_t d_out, int64_t d_in,
                               int64_t M, size_t *bytes)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!bytes) return BSQ_ERR_ARG;
    if ((s = check_shape(*cfg, d_out, d_in)) != BSQ_OK) return s;
    if (n_mats < 1) return BSQ_ERR_ARG;
    switch (op) {
    case BSQ_OP_ENCODE: *bytes = encode_ws_layout(*cfg, n_mats, d_out, d_in, nullptr, nullptr); return BSQ_OK;
    case BSQ_OP_GEMV:
        if (n_mats > BSQ_MAX_GROUP) return BSQ_ERR_ARG;
        *bytes = gemv_ws_bytes(coded_cfg(*cfg), n_mats, d_out, d_in);
        return BSQ_OK;
    case BSQ_OP_GEMM:
        if (M < 0) return BSQ_ERR_ARG;
        *bytes = gemm_ws_bytes(coded_cfg(*cfg), d_out, d_in, M);
        return BSQ_OK;
    case BSQ_OP_SELECT:
        if (n_mats != 1) return BSQ_ERR_ARG;
        *bytes = select_ws_layout(d_out, nullptr, nullptr);
        return BSQ_OK;
    default: return BSQ_ERR_ARG;
    }
}

bsq_status bsq_codec_bytes(const bsq_config *cfg, size_t *bytes)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!bytes) return BSQ_ERR_ARG;
    *bytes = codec_total_bytes(*cfg);
    return BSQ_OK;
}

bsq_status bsq_codec_prepare(const bsq_config *cfg, const bsq_decoder *dec, void *codec, size_t codec_bytes,
                             void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!codec) return BSQ_ERR_ARG;
    if (!aligned(codec, 256)) return BSQ_ERR_ALIGN;
    if (codec_bytes < codec_total_bytes(*cfg)) return BSQ_ERR_BUFFER_TOO_SMALL;
    if (cfg->dec_kind != BSQ_DEC_IDENTITY) {
        if (!dec) return BSQ_ERR_ARG;
        for (int i = 0; i < cfg->stages; ++i) {
            if (!dec[i].W1 || !dec[i].b1) return BSQ_ERR_ARG;
            if ((cfg->dec_kind == BSQ_DEC_MLP || cfg->dec_kind == BSQ_DEC_MLP_RES1) && (!dec[i].W2 || !dec[i].b2))
                return BSQ_ERR_ARG;
            if (cfg->dec_kind == BSQ_DEC_MLP_RES1 && (!dec[i].R || !dec[i].c)) return BSQ_ERR_ARG;
        }
    }
    if (cfg->encoder == BSQ_ENC_LINEAR) {
        if (!dec) return BSQ_ERR_ARG;
        for (int i = 0; i < cfg->stages; ++i)
            if (!dec[i].E) return BSQ_ERR_ARG;
    }
    bsq_decoder none[BSQ_MAX_STAGES] = {};
    return from_hip(launch_codec_tables(*cfg, dec ? dec : none, codec, static_cast<hipStream_t>(stream)));
}

namespace {

bsq_status encode_common(const bsq_config *cfg, const void *codec, const void *W, int32_t w_dtype, int64_t n_mats,
                         int64_t d_out, int64_t d_in, const float *g, const int32_t *given, const bsq_layer *out,
                         int32_t *err, void *ws, size_t ws_bytes, void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    const bsq_config &c = *cfg;
    if (!codec || !out || !err || !ws) return BSQ_ERR_ARG;
    if (!W && d_out > 0) return BSQ_ERR_ARG;
    if (w_dtype != BSQ_F32 && w_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if ((s = check_shape(c, d_out, d_in)) != BSQ_OK) return s;
    if (n_mats < 1) return BSQ_ERR_ARG;
    if ((s = check_layer(c, out, true, !row_axis(c))) != BSQ_OK) return s;
    if (out->d_out != d_out || out->d_in != d_in || out->n_mats != n_mats) return BSQ_ERR_ARG;
    if (!aligned(W, 16) || !aligned(codec, 256) || !aligned(ws, 256) || !aligned(err, 4)) return BSQ_ERR_ALIGN;
    if (out->k > 0 && d_in > (int64_t(1) << 18)) return BSQ_ERR_UNSUPPORTED;
    // the TopK (and the set check) keeps one bit per channel of the axis in LDS
    if (out->k > 0 && row_axis(c) && d_out > (int64_t(1) << 18)) return BSQ_ERR_UNSUPPORTED;
    // the protected-row pass runs one block per (row, matrix), matrices along grid y
    if (out->k > 0 && row_axis(c) && n_mats > 65535) return BSQ_ERR_UNSUPPORTED;
    if (g && !aligned(g, 4)) return BSQ_ERR_ALIGN;
    if (given && out->k > 0 && !aligned(given, 4)) return BSQ_ERR_ALIGN;
    const size_t need = encode_ws_layout(c, n_mats, d_out, d_in, nullptr, nullptr);
    if (ws_bytes < need) return BSQ_ERR_BUFFER_TOO_SMALL;
    EncodeWs w{};
    encode_ws_layout(c, n_mats, d_out, d_in, static_cast<char *>(ws), &w);
    return from_hip(launch_encode(c, codec, W, w_dtype, n_mats, d_out, d_in, g, given, *out, err, w,
                                  static_cast<hipStream_t>(stream)));
}

}  // namespace

bsq_status bsq_encode(const bsq_config *cfg, const void *codec, const void *W, int32_t w_dtype, int64_t n_mats,
                      int64_t d_out, int64_t d_in, const float *g, const bsq_layer *out, int32_t *err, void *ws,
                      size_t ws_bytes, void *stream)
{
    return encode_common(cfg, codec, W, w_dtype, n_mats, d_out, d_in, g, nullptr, out, err, ws, ws_bytes, stream);
}

bsq_status bsq_encode_with_set(const bsq_config *cfg, const void *codec, const void *W, int32_t w_dtype,
                               int64_t n_mats, int64_t d_out, int64_t d_in, const int32_t *idx, const bsq_layer *out,
                               int32_t *err, void *ws, size_t ws_bytes, void *stream)
{
    if (!cfg) return BSQ_ERR_ARG;
    if (cfg->protect_num > 0 && !idx && k_of(*cfg, d_out, d_in) > 0) return BSQ_ERR_ARG;
    return encode_common(cfg, codec, W, w_dtype, n_mats, d_out, d_in, nullptr, idx, out, err, ws, ws_bytes,
                         stream);
}

bsq_status bsq_coupled_select(const bsq_config *cfg, const void *W_gate, const void *W_up, const void *W_down,
                              int32_t w_dtype, int64_t d_model, int64_t d_ffn, const float *g_gate,
                              const float *g_up, const float *g_down, int32_t *idx, double *scores, int32_t *err,
                              void *ws, size_t ws_bytes, void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (w_dtype != BSQ_F32 && w_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if (d_model < 1 || d_ffn < 1) return BSQ_ERR_SHAPE;
    // fp64 partial norms of whole columns/rows, one lane each; the TopK bitmap in LDS
    if (d_ffn > (int64_t(1) << 18) || d_model > (int64_t(1) << 31)) return BSQ_ERR_UNSUPPORTED;
    if (!W_gate || !W_up || !W_down || !err || !ws) return BSQ_ERR_ARG;
    const int64_t k = (cfg->protect_num == 0) ? 0 : (d_ffn * cfg->protect_num + cfg->protect_den - 1) / cfg->protect_den;
    if (k > 0 && !idx) return BSQ_ERR_ARG;
    if (!aligned(W_gate, 16) || !aligned(W_up, 16) || !aligned(W_down, 16) || !aligned(err, 4) || !aligned(ws, 256))
        return BSQ_ERR_ALIGN;
    if ((g_gate && !aligned(g_gate, 4)) || (g_up && !aligned(g_up, 4)) || (g_down && !aligned(g_down, 4)))
        return BSQ_ERR_ALIGN;
    if ((idx && !aligned(idx, 4)) || (scores && !aligned(scores, 8))) return BSQ_ERR_ALIGN;
    if (ws_bytes < select_ws_layout(d_ffn, nullptr, nullptr)) return BSQ_ERR_BUFFER_TOO_SMALL;
    SelectWs w{};
    select_ws_layout(d_ffn, static_cast<char *>(ws), &w);
    return from_hip(launch_coupled_select(W_gate, W_up, W_down, w_dtype, d_model, d_ffn, g_gate, g_up, g_down, k, idx,
                                          scores, err, w, static_cast<hipStream_t>(stream)));
}

bsq_status bsq_decode(const bsq_config *cfg, const void *codec, const bsq_layer *layer, void *W_hat,
                      int32_t out_dtype, void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!codec || !layer) return BSQ_ERR_ARG;
    if (!W_hat && layer->d_out > 0) return BSQ_ERR_ARG;
    if (out_dtype != BSQ_F32 && out_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if ((s = check_layer(*cfg, layer, true, false)) != BSQ_OK) return s;
    if (!aligned(W_hat, 16) || !aligned(codec, 256)) return BSQ_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bsq_layer coded = coded_layer(*cfg, *layer);
    if ((s = from_hip(launch_decode(coded_cfg(*cfg), codec, coded, W_hat, out_dtype, st))) != BSQ_OK) return s;
    if (!row_axis(*cfg)) return BSQ_OK;
    return from_hip(launch_decode_rows(*layer, cfg->protect_format, W_hat, out_dtype, st));
}

bsq_status bsq_decode_stage(const bsq_config *cfg, const void *codec, const bsq_layer *layer, int32_t stage,
                            int32_t accumulate, void *W_hat, void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!codec || !layer) return BSQ_ERR_ARG;
    if (!W_hat && layer->d_out > 0) return BSQ_ERR_ARG;
    if (stage < 0 || stage >= cfg->stages || (accumulate != 0 && accumulate != 1)) return BSQ_ERR_ARG;
    if ((s = check_layer(*cfg, layer, true, false)) != BSQ_OK) return s;
    if (!aligned(W_hat, 16) || !aligned(codec, 256)) return BSQ_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bsq_layer coded = coded_layer(*cfg, *layer);
    if ((s = from_hip(launch_decode_stage(coded_cfg(*cfg), codec, coded, stage, accumulate, W_hat, st))) != BSQ_OK)
        return s;
    if (!row_axis(*cfg) || stage != cfg->stages - 1) return BSQ_OK;
    return from_hip(launch_decode_rows(*layer, cfg->protect_format, W_hat, BSQ_F32, st));
}

namespace {

bsq_status check_gemv(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                      const bsq_lora *loras, int32_t x_dtype, void *const *y, int32_t y_dtype, void *ws,
                      size_t ws_bytes)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (n < 1 || n > BSQ_MAX_GROUP) return BSQ_ERR_ARG;
    if (!layers || !ws) return BSQ_ERR_ARG;
    if (x_dtype != BSQ_F32 && x_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if (y && y_dtype != BSQ_F32 && y_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    for (int m = 0; m < n; ++m) {
        if ((s = check_layer(*cfg, &layers[m], codecs != nullptr, codecs != nullptr)) != BSQ_OK) return s;
        if (layers[m].n_mats != 1 || layers[m].d_in != layers[0].d_in) return BSQ_ERR_ARG;
        if (codecs) {
            if (!codecs[m]) return BSQ_ERR_ARG;
            if (!aligned(codecs[m], 256)) return BSQ_ERR_ALIGN;
        }
        if (y) {
            if (!y[m] && layers[m].d_out > 0) return BSQ_ERR_ARG;
            if (!aligned(y[m], y_dtype == BSQ_F32 ? 4 : 2)) return BSQ_ERR_ALIGN;
        }
        if (loras && (s = check_lora(&loras[m])) != BSQ_OK) return s;
    }
    if (!aligned(ws, 256)) return BSQ_ERR_ALIGN;
    // the d = 16 streaming kernel (decoders other than the width-16 symmetric
    // one) holds one 128-input segment per thread of a 512-thread block
    const bool split16 = codec_has_split(*cfg) && cfg->hidden == 16;
    if (x_dtype == BSQ_BF16 && cfg->d == 16 && cfg->b == 16 && !split16 && layers[0].pitch * cfg->d / 128 > 512)
        return BSQ_ERR_UNSUPPORTED;
    if (x_dtype == BSQ_BF16 && !row_axis(*cfg) && layers[0].k > 4096) return BSQ_ERR_UNSUPPORTED;
    int64_t max_d_out = 0;
    for (int m = 0; m < n; ++m) max_d_out = layers[m].d_out > max_d_out ? layers[m].d_out : max_d_out;
    if (ws_bytes < gemv_ws_bytes(coded_cfg(*cfg), n, max_d_out, layers[0].d_in)) return BSQ_ERR_BUFFER_TOO_SMALL;
    return BSQ_OK;
}

// the layers as the streaming kernels see them (coded_layer of each)
struct CodedGroup {
    bsq_layer L[BSQ_MAX_GROUP];
    CodedGroup(const bsq_config &c, int n, const bsq_layer *layers)
    {
        for (int m = 0; m < n; ++m) L[m] = coded_layer(c, layers[m]);
    }
};

}  // namespace

bsq_status bsq_gemv_prepare(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                            const bsq_lora *loras, const void *x, int32_t x_dtype, void *ws, size_t ws_bytes,
                            void *stream)
{
    bsq_status s = check_gemv(cfg, n, codecs, layers, loras, x_dtype, nullptr, BSQ_F32, ws, ws_bytes);
    if (s != BSQ_OK) return s;
    if (!x) return BSQ_ERR_ARG;
    if (!aligned(x, x_dtype == BSQ_F32 ? 4 : 2)) return BSQ_ERR_ALIGN;
    // the d = 16 symmetric decoder folds its output layer into x here
    if (!codecs && codec_has_split(*cfg) && x_dtype == BSQ_BF16) return BSQ_ERR_ARG;
    const CodedGroup g(*cfg, n, layers);
    return from_hip(launch_gemv_prep(coded_cfg(*cfg), n, codecs, g.L, loras, x, x_dtype, ws, false,
                                     static_cast<hipStream_t>(stream)));
}

bsq_status bsq_gemv_run(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                        const bsq_lora *loras, const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                        void *ws, size_t ws_bytes, int32_t *err, void *stream)
{
    if (!codecs || !y || !x) return BSQ_ERR_ARG;
    bsq_status s = check_gemv(cfg, n, codecs, layers, loras, x_dtype, y, y_dtype, ws, ws_bytes);
    if (s != BSQ_OK) return s;
    if (!aligned(x, x_dtype == BSQ_F32 ? 4 : 16)) return BSQ_ERR_ALIGN;
    if (err && !aligned(err, 4)) return BSQ_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const CodedGroup g(*cfg, n, layers);
    if ((s = from_hip(launch_gemv_run(coded_cfg(*cfg), n, codecs, g.L, loras, x, x_dtype, y, y_dtype, ws, false,
                                      err, st))) != BSQ_OK)
        return s;
    if (!row_axis(*cfg)) return BSQ_OK;
    return from_hip(launch_gemv_rows(n, layers, cfg->protect_format, loras, x, x_dtype, y, y_dtype, st));
}

namespace {

// bsq_gemv after validation, on a workspace of one configuration or on the
// shared scratch array (scratch_layout)
bsq_status gemv_launch(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                       const bsq_lora *loras, const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                       void *ws, bool scratch_layout, int32_t *err, hipStream_t st)
{
    bsq_status s;
    const bsq_config cc = coded_cfg(*cfg);
    const CodedGroup g(*cfg, n, layers);
    if ((s = from_hip(launch_gemv_prep(cc, n, codecs, g.L, loras, x, x_dtype, ws, scratch_layout, st))) != BSQ_OK)
        return s;
    if ((s = from_hip(launch_gemv_run(cc, n, codecs, g.L, loras, x, x_dtype, y, y_dtype, ws, scratch_layout, err,
                                      st))) != BSQ_OK)
        return s;
    if (!row_axis(*cfg)) return BSQ_OK;
    return from_hip(launch_gemv_rows(n, layers, cfg->protect_format, loras, x, x_dtype, y, y_dtype, st));
}

}  // namespace

bsq_status bsq_gemv(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                    const bsq_lora *loras, const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                    void *ws, size_t ws_bytes, int32_t *err, void *stream)
{
    if (!codecs || !y || !x) return BSQ_ERR_ARG;
    bsq_status s = check_gemv(cfg, n, codecs, layers, loras, x_dtype, y, y_dtype, ws, ws_bytes);
    if (s != BSQ_OK) return s;
    if (!aligned(x, x_dtype == BSQ_F32 ? 4 : 16)) return BSQ_ERR_ALIGN;
    if (err && !aligned(err, 4)) return BSQ_ERR_ALIGN;
    return gemv_launch(cfg, n, codecs, layers, loras, x, x_dtype, y, y_dtype, ws, false, err,
                       static_cast<hipStream_t>(stream));
}

bsq_status bsq_gemv_noalloc(const bsq_config *cfg, int32_t n, const void *const *codecs, const bsq_layer *layers,
                            const bsq_lora *loras, const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                            int32_t clear_scratch, int32_t *err, void *stream)
{
    if (!codecs || !y || !x || !layers) return BSQ_ERR_ARG;
    if (clear_scratch != 0 && clear_scratch != 1) return BSQ_ERR_ARG;
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (n < 1 || n > BSQ_MAX_GROUP) return BSQ_ERR_ARG;
    int64_t max_d_out = 0;
    for (int m = 0; m < n; ++m) {
        if ((s = check_shape(*cfg, layers[m].d_out, layers[m].d_in)) != BSQ_OK) return s;
        max_d_out = layers[m].d_out > max_d_out ? layers[m].d_out : max_d_out;
    }
    // the group's workspace must fit the library's scratch array
    if (!gemv_scratch_fits(coded_cfg(*cfg), n, max_d_out, layers[0].d_in)) return BSQ_ERR_BUFFER_TOO_SMALL;
    // everything bsq_gemv validates, with the array standing in for the
    // workspace (it is 256-byte aligned and large enough)
    if ((s = check_gemv(cfg, n, codecs, layers, loras, x_dtype, y, y_dtype, reinterpret_cast<void *>(uintptr_t(256)),
                        size_t(BSQ_GEMV_NOALLOC_SCRATCH_BYTES))) != BSQ_OK)
        return s;
    if (!aligned(x, x_dtype == BSQ_F32 ? 4 : 16)) return BSQ_ERR_ALIGN;
    if (err && !aligned(err, 4)) return BSQ_ERR_ALIGN;
    hipStream_t st = static_cast<hipStream_t>(stream);
    void *ws = nullptr;
    if ((s = from_hip(gemv_scratch(clear_scratch != 0, &ws, st))) != BSQ_OK) return s;
    return gemv_launch(cfg, n, codecs, layers, loras, x, x_dtype, y, y_dtype, ws, true, err, st);
}

bsq_status bsq_gemm(const bsq_config *cfg, const void *codec, const bsq_layer *layer, const bsq_lora *lora,
                    const void *X, int32_t x_dtype, int64_t M, int64_t ldx, void *Y, int32_t y_dtype, int64_t ldy,
                    void *ws, size_t ws_bytes, int32_t *err, void *stream)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!codec || !ws || !layer) return BSQ_ERR_ARG;
    if (M > 0 && (!X || (!Y && layer->d_out > 0))) return BSQ_ERR_ARG;
    if (x_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if (y_dtype != BSQ_F32 && y_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if ((s = check_layer(*cfg, layer, true, false)) != BSQ_OK) return s;
    if (layer->n_mats != 1) return BSQ_ERR_ARG;
    if ((s = check_lora(lora)) != BSQ_OK) return s;
    if (M < 0 || ldx < layer->d_in || ldy < layer->d_out || ldx % 8 != 0) return BSQ_ERR_SHAPE;
    if (!aligned(X, 16) || !aligned(ws, 256) || !aligned(codec, 256)) return BSQ_ERR_ALIGN;
    if (!aligned(Y, y_dtype == BSQ_F32 ? 4 : 2)) return BSQ_ERR_ALIGN;
    if (err && !aligned(err, 4)) return BSQ_ERR_ALIGN;
    const bsq_config cc = coded_cfg(*cfg);
    if (ws_bytes < gemm_ws_bytes(cc, layer->d_out, layer->d_in, M)) return BSQ_ERR_BUFFER_TOO_SMALL;
    const bool rows = row_axis(*cfg);
    if (!rows && layer->k > 4096) return BSQ_ERR_UNSUPPORTED;
    // the protected-row launch takes four tokens per block along grid y
    if (rows && (M + 3) / 4 > 65535) return BSQ_ERR_UNSUPPORTED;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bsq_layer coded = coded_layer(*cfg, *layer);
    if ((s = from_hip(launch_gemm(cc, codec, coded, lora, X, M, ldx, Y, y_dtype, ldy, ws, err, st))) != BSQ_OK)
        return s;
    if (!rows) return BSQ_OK;
    return from_hip(launch_gemm_rows(*layer, cfg->protect_format, lora, X, M, ldx, Y, y_dtype, ldy, gemm_lora_t(ws), st));
}


namespace {
bsq_status check_train_cfg(const bsq_config *cfg)
{
    bsq_status s = check_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (cfg->encoder != BSQ_ENC_LINEAR || cfg->dec_kind != BSQ_DEC_MLP) return BSQ_ERR_UNSUPPORTED;
    return BSQ_OK;
}

bool finite_hparams(const bsq_train_hparams *hp)
{
    const float v[8] = {hp->lambda_c, hp->lambda_e, hp->gamma, hp->tau, hp->lr, hp->beta1, hp->beta2, hp->eps};
    for (float f : v)
        if (!(f == f) || f > 3.0e38f || f < -3.0e38f) return false;
    return hp->beta1 >= 0.0f && hp->beta1 < 1.0f && hp->beta2 >= 0.0f && hp->beta2 < 1.0f && hp->eps >= 0.0f;
}
}  // namespace

bsq_status bsq_train_param_count(const bsq_config *cfg, int64_t *count)
{
    bsq_status s = check_train_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!count) return BSQ_ERR_ARG;
    *count = train_param_count(*cfg);
    return BSQ_OK;
}

bsq_status bsq_train_workspace_bytes(const bsq_config *cfg, int64_t n, size_t *bytes)
{
    bsq_status s = check_train_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!bytes || n < 1) return BSQ_ERR_ARG;
    if (n > (int64_t(1) << 26)) return BSQ_ERR_UNSUPPORTED;
    *bytes = train_ws_bytes(*cfg, n);
    return BSQ_OK;
}

bsq_status bsq_train_grad(const bsq_config *cfg, const bsq_train_hparams *hp, const void *chunks, int32_t x_dtype,
                          int64_t n_total, const int64_t *idx, int64_t n, const float *theta, float *grad,
                          float *loss, int32_t *err, void *ws, size_t ws_bytes, void *stream)
{
    bsq_status s = check_train_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!hp || !chunks || !theta || !grad || !loss || !ws) return BSQ_ERR_ARG;
    if (!finite_hparams(hp)) return BSQ_ERR_ARG;
    if (x_dtype != BSQ_F32 && x_dtype != BSQ_BF16) return BSQ_ERR_DTYPE;
    if (n < 1 || n_total < 1 || (!idx && n > n_total)) return BSQ_ERR_SHAPE;
    if (n > (int64_t(1) << 26)) return BSQ_ERR_UNSUPPORTED;
    if (!aligned(chunks, x_dtype == BSQ_F32 ? 4 : 2) || !aligned(theta, 4) || !aligned(grad, 4) ||
        !aligned(loss, 4) || !aligned(ws, 256) || (idx && !aligned(idx, 8)) || (err && !aligned(err, 4)))
        return BSQ_ERR_ALIGN;
    if (ws_bytes < train_ws_bytes(*cfg, n)) return BSQ_ERR_BUFFER_TOO_SMALL;
    return from_hip(launch_train_grad(*cfg, *hp, chunks, x_dtype, n_total, idx, n, theta, grad, loss, err, ws,
                                      static_cast<hipStream_t>(stream)));
}

bsq_status bsq_train_adam(const bsq_config *cfg, const bsq_train_hparams *hp, int32_t step, float *theta,
                          const float *grad, float *m, float *v, void *stream)
{
    bsq_status s = check_train_cfg(cfg);
    if (s != BSQ_OK) return s;
    if (!hp || !theta || !grad || !m || !v || step < 1) return BSQ_ERR_ARG;
    if (!finite_hparams(hp)) return BSQ_ERR_ARG;
    if (!aligned(theta, 4) || !aligned(grad, 4) || !aligned(m, 4) || !aligned(v, 4)) return BSQ_ERR_ALIGN;
    return from_hip(launch_train_adam(*cfg, *hp, step, theta, grad, m, v, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
