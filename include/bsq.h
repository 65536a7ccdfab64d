/*
 * bsq.h -- C ABI of libbsq.so, an MI355X (gfx950) implementation of the
 * binary spherical (BSQ) weight codec of BiSCo-LLM and of the products that
 * consume its bit-packed sign streams.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers named "device" point into GPU memory owned by the caller; the
 *   library never allocates, frees or retains memory. Host structs are read
 *   during the call only.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   Every entry point that launches work is asynchronous on that stream.
 * - Arguments are validated on the host before anything is launched; a
 *   non-BSQ_OK return means nothing was enqueued. Device-side conditions are
 *   reported through a device error word (int32, caller-owned, zeroed by the
 *   caller) into which the kernels OR the BSQ_DEVERR_* bits below; the caller
 *   reads it after synchronising.
 * - No C++ exception crosses this boundary.
 * - Calls are re-entrant; two calls that share an output or workspace buffer
 *   on different streams race.
 *
 * Data layout of an encoded matrix W [d_out][d_in] (row-major)
 * ------------------------------------------------------------
 * chunk (i, c) = W[i, c*d : (c+1)*d], C = d_in / d chunks per row, every
 * row is padded to `pitch` = roundup(C, 16) chunks and the rows to a
 * multiple of 64 (padding: code 0, gain +0). The code and gain planes are
 * stored in 64-row x 16-chunk tiles:
 *   element (i, c) is at ((i/64 * pitch/16 + c/16) * 64 + i%64) * 16 + c%16
 * i.e. [ceil(d_out/64)][pitch/16][64][16], so that 64 rows x 16 chunks are one
 * contiguous 1 KiB (d = 8) or 2 KiB (d = 16) code tile and 2 KiB gain tile.
 *   codes[s]   uint8 (b = 8) or uint16 little-endian (b = 16), tiled:
 *              bit m of a code is 1 iff element m of the encoder output z
 *              is >= 0 (+0 and -0 give 1), element m -> bit m (LSB first);
 *              z is the stage target itself with the identity encoder;
 *   gains[s]   fp16 bits, tiled: per-chunk least-squares gain of
 *              stage s (round to nearest even, finite overflow saturated);
 *   prot_idx   int32 [k], the protected input columns in ascending order;
 *   prot_q8    8-bit [d_out][kp], kp = roundup(k, 16), 16-byte aligned:
 *              row i holds the stored bytes of row i's k protected entries
 *              (format by protect_format: symmetric int8, or FP8-E4M3 /
 *              FP8-E5M2), then kp - k zero bytes;
 *   prot_scale fp32  [k], one scale per protected column;
 *   prot_bits  uint32 [pitch * d / 32], bit j%32 of word j/32 set iff input
 *              column j is protected (the same set as prot_idx, as a bitmap
 *              over the padded columns; padding bits 0). Derived metadata
 *              written by bsq_encode so that the products can mask the
 *              activations with one scalar load per 128 columns.
 * A stack of n_mats matrices of one shape stores these arrays back to back,
 * matrix-major ([n_mats][...]).
 *
 * With protect_axis = 1 (protected output rows, the output-channel axis of
 * the protection-axis ablation in Section IV-D, and the gate/up side of
 * eq. mlp_coupled_protection) the protected slices are k whole rows:
 *   prot_idx   int32 [k], the protected rows in ascending order;
 *   prot_q8    8-bit [k][q8_pitch(d_in)], q8_pitch(n) = roundup(n, 16):
 *              row p holds the stored bytes of row prot_idx[p], then zero
 *              bytes;
 *   prot_scale fp32  [k], one scale per protected row;
 *   prot_bits  unused (may be NULL);
 * and the protected rows are not BSQ-coded: their code and gain planes hold
 * code 0 and gain +0. k = ceil(rho * d_out) for this axis.
 */
#ifndef BSQ_H
#define BSQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BSQ_ABI_VERSION 8
#define BSQ_MAX_STAGES 4
#define BSQ_PITCH_ALIGN 16
#define BSQ_MAX_HIDDEN 64
#define BSQ_MAX_LORA_RANK 16
#define BSQ_MAX_GROUP 8
/* size of the library-owned workspace of bsq_gemv_noalloc, per GPU */
#define BSQ_GEMV_NOALLOC_SCRATCH_BYTES (8u << 20)

typedef enum {
    BSQ_OK = 0,
    BSQ_ERR_ARG = 1,              /* null pointer or value out of range */
    BSQ_ERR_SHAPE = 2,            /* d_in not a multiple of d, empty where not allowed, ... */
    BSQ_ERR_DTYPE = 3,            /* unsupported element type for this argument */
    BSQ_ERR_ALIGN = 4,            /* a buffer is not aligned as documented */
    BSQ_ERR_BUFFER_TOO_SMALL = 5, /* workspace or codec buffer smaller than required */
    BSQ_ERR_NONFINITE = 6,        /* bit 0 of a device error word: NaN/Inf in the input */
    BSQ_ERR_DEVICE = 7,           /* a HIP launch or runtime call failed */
    BSQ_ERR_UNSUPPORTED = 8       /* valid configuration that this build does not implement */
} bsq_status;

/* Bits of a device error word.
 *   NONFINITE  the weights hold NaN or Inf (bsq_encode, bsq_encode_with_set,
 *              bsq_coupled_select);
 *   BAD_SET    a given protected set is not strictly ascending or out of
 *              range (bsq_encode_with_set);
 *   TIMEOUT    a GEMV's finishing workgroup gave up waiting for another
 *              workgroup's partial result (never expected: workgroups run in
 *              dispatch order, and the wait is bounded only so that a fault
 *              elsewhere cannot hang the queue). The affected outputs are NaN
 *              and the workspace is left POISONED;
 *   POISONED   the workspace was marked by an earlier call that timed out: a
 *              late partial may still sit in it, so nothing in it was used
 *              and the outputs of this call are NaN. Zero-fill the workspace
 *              (after synchronising) to use it again. */
#define BSQ_DEVERR_NONFINITE 1
#define BSQ_DEVERR_BAD_SET 2
#define BSQ_DEVERR_TIMEOUT 4
#define BSQ_DEVERR_POISONED 8

typedef enum { BSQ_F32 = 0, BSQ_BF16 = 1 } bsq_dtype;

/* Decoder families of the paper's codec ablation (Section IV-D, Table
 * "BSQ codec components"): identity (y = q), linear, and the compact
 * symmetric decoder with no residual block (one hidden ReLU layer) or with
 * one residual block on its hidden layer. */
typedef enum {
    BSQ_DEC_IDENTITY = 0,
    BSQ_DEC_LINEAR = 1,
    BSQ_DEC_MLP = 2,
    BSQ_DEC_MLP_RES1 = 3
} bsq_dec_kind;

/* Storage format of the protected path (Table "BSQ codec components": INT8,
 * FP8-E4M3, FP8-E5M2). One byte per protected element and one fp32 scale per
 * protected slice; the element's weight is value(byte) * scale, and the
 * scale is the slice's largest magnitude over the format's largest finite
 * value (127, 448, 57344).
 *   INT8: two's complement, round half to even, clamped to +-127;
 *   E4M3: sign, 4 exponent bits (bias 7), 3 fraction bits, subnormals, no
 *         infinities (S.1111.111 is NaN);
 *   E5M2: sign, 5 exponent bits (bias 15), 2 fraction bits, subnormals,
 *         S.11111.00 is infinity.
 * FP8 rounding: nearest finite value, ties to the even code, sign kept (a
 * negative value that rounds to zero stores -0), magnitudes past the largest
 * finite value store it. */
typedef enum { BSQ_PROT_INT8 = 0, BSQ_PROT_E4M3 = 1, BSQ_PROT_E5M2 = 2 } bsq_prot_format;

/* The encoder E_phi of Section III-C, which maps a chunk (or a stage's
 * residual target) r in R^d to the latent z in R^b whose signs are the code:
 *   IDENTITY: z = r (requires b = d);
 *   LINEAR:   z = E r with a learned E [b][d] per stage; z_m is the fp32
 *             fmaf chain sum_j E[m][j] r_j from +0, j in order.
 * With the linear encoder b may differ from d (codebook_bits and
 * codebook_dim of Section III-A, e.g. the b/d = 2 settings of Section
 * III-D). */
typedef enum { BSQ_ENC_IDENTITY = 0, BSQ_ENC_LINEAR = 1 } bsq_enc_kind;

typedef struct {
    int32_t d;           /* chunk length: 8 or 16 (Section III-A, codebook_dim) */
    int32_t b;           /* code bits per stage: 8 or 16 (codebook_bits); b = d unless the encoder is LINEAR */
    int32_t stages;      /* residual stages S, 1..4 (Section III-D; default 2) */
    int32_t dec_kind;    /* bsq_dec_kind */
    int32_t hidden;      /* hidden width h of the symmetric decoders, 1..64; ignored for other kinds */
    int32_t protect_num; /* protected-channel ratio rho = num/den (eq. protected_channel_selection); */
    int32_t protect_den; /*   num = 0 disables the protected path; k = ceil(n*num/den) for the n */
                         /*   channels of the protected axis (d_in for columns, d_out for rows) */
    int32_t protect_axis; /* 0: protected input columns; 1: protected output rows */
    int32_t protect_format; /* bsq_prot_format of the protected payload */
    int32_t encoder;        /* bsq_enc_kind */
} bsq_config;

/* Parameters of one stage's codec, fp32, row-major, device pointers: the
 * encoder E [b][d] (LINEAR encoder only, else unused) and the decoder.
 *   MLP:      W1 [h][b], b1 [h], W2 [d][h], b2 [d];
 *             y = W2 relu(W1 q + b1) + b2, relu(a) = a > 0 ? a : +0
 *   MLP_RES1: the MLP's tensors and R [h][h], c [h];
 *             a = relu(W1 q + b1); a' = a + relu(R a + c); y = W2 a' + b2
 *   LINEAR:   W1 = M [d][b], b1 = beta [d]; y = M q + beta   (W2, b2 unused)
 *   IDENTITY: y = q                                           (all unused)
 * with q_j = +-1/sqrt(b) (Section III-C, sphere map and sign binarisation).
 * Every dot product is an fp32 fmaf chain from the bias, in index order; R
 * and c may be NULL for the other kinds. */
typedef struct {
    const float *W1;
    const float *b1;
    const float *W2;
    const float *b2;
    const float *R;
    const float *c;
    const float *E;
} bsq_decoder;

/* One encoded matrix (or a stack of n_mats of one shape), device pointers.
 * prot_* may be NULL when k == 0; bsq_decode and bsq_gemm do not read
 * prot_bits (they may receive NULL there). */
typedef struct {
    void *codes[BSQ_MAX_STAGES];
    uint16_t *gains[BSQ_MAX_STAGES];
    int32_t *prot_idx;
    int8_t *prot_q8;     /* stored bytes in the config's protect_format */
    float *prot_scale;
    uint32_t *prot_bits;
    int64_t d_out;
    int64_t d_in;
    int64_t pitch;   /* chunks per row including padding: roundup(d_in/d, 16) */
    int64_t k;       /* protected columns per matrix */
    int64_t n_mats;  /* matrices stored back to back; 1 for a single matrix */
} bsq_layer;

/* Optional LoRA compensation term y += B (A x) (Section III-F). bf16,
 * device pointers: A [rank][d_in], B [d_out][rank]; rank 1..16. */
typedef struct {
    const uint16_t *A;
    const uint16_t *B;
    int32_t rank;
} bsq_lora;

/* Storage accounting of eq. real_size for one matrix:
 * S_tot = S_code + S_dec + S_8bit + S_LoRA + S_meta (bytes). S_dec counts the
 * stage decoders (and a linear encoder's b d parameters) once (a model counts
 * them once per category, because every layer of a category shares them).
 * Buffer sizes include the row padding; a code plane holds b / 8 bytes per
 * chunk. */
typedef struct {
    int64_t pitch;
    int64_t k;
    int64_t chunks;             /* d_out * d_in / d */
    int64_t code_plane_bytes;   /* one stage's code buffer, padded */
    int64_t gain_plane_bytes;   /* one stage's gain buffer, padded */
    int64_t idx_bytes, q8_bytes, scale_bytes;  /* q8_bytes = d_out * roundup(k, 16) */
    int64_t bits_bytes;         /* prot_bits (0 when k == 0); not part of S_tot */
    double S_code, S_dec, S_8bit, S_LoRA, S_meta, S_tot;
    double bpw_nominal;         /* S * b / d (Section III-A) */
    double bpw_real;            /* 8 * S_tot / (d_out * d_in) */
} bsq_sizes;

/* Operations for bsq_workspace_bytes. BSQ_OP_SELECT is bsq_coupled_select,
 * with d_out = d_ffn and d_in = d_model. */
typedef enum { BSQ_OP_ENCODE = 0, BSQ_OP_GEMV = 1, BSQ_OP_GEMM = 2, BSQ_OP_SELECT = 3 } bsq_op;

/* ---------------------------------------------------------------------- */

/* Library ABI version (BSQ_ABI_VERSION). */
int32_t bsq_version(void);

/* Testing aid: the number of polls a GEMV's finishing workgroup makes for
 * another workgroup's partial result before it gives up (BSQ_DEVERR_TIMEOUT;
 * bsq_gemm has no such wait).
 * 0 makes every such wait give up at once, so that the timeout and poison
 * handling can be exercised with every kernel still exiting normally; a
 * negative value restores the default (about a second of polling). Applies
 * to calls issued afterwards (a captured graph keeps the value it was
 * captured with); process-wide, host only. Returns the previous value. */
int32_t bsq_debug_set_wait_limit(int32_t polls);

/* Static description of a status code; never NULL. */
const char *bsq_status_str(int32_t status);

/* Validate a configuration (host only, launches nothing). */
bsq_status bsq_config_check(const bsq_config *cfg);

/* Sizes of the encoded buffers and the eq. real_size accounting for one
 * d_out x d_in matrix with an optional LoRA of the given rank (0 = none).
 * Host only. */
bsq_status bsq_layer_sizes(const bsq_config *cfg, int64_t d_out, int64_t d_in,
                           int32_t lora_rank, bsq_sizes *out);

/* Bytes of device workspace an operation needs (host only). For ENCODE,
 * n_mats is the stack size and M is ignored; for GEMV n_mats is the group
 * size; for GEMM M is the number of tokens. */
bsq_status bsq_workspace_bytes(const bsq_config *cfg, int32_t op, int64_t n_mats,
                               int64_t d_out, int64_t d_in, int64_t M, size_t *bytes);

/* A prepared codec: the stage decoders evaluated on all 2^b codes
 * (Section III-G, batched parallel residual decoding needs only D_s(code)).
 * The buffer holds, per stage, an fp32 table [2^b][d] filled in the same fp32
 * operation order as the encoder's definition (so encode and decode are
 * exact), then a bf16 copy [2^b][d] for the GEMV's products and an fp16 copy
 * [2^b][d] for the GEMM's decode (both rounded to nearest even). For the
 * symmetric decoder at d = 16 it also holds, per stage, the hidden
 * pre-activation W1 q + b1 split by code byte (two fp16 tables [256][h] whose
 * entries add up to it) and copies of W2 and b2, from which the GEMV
 * evaluates that decoder. One codec per (category, stage set) serves every
 * layer of that category.
 * bsq_codec_bytes: required size (host only).
 * bsq_codec_prepare: `dec` is a host array of `stages` bsq_decoder structs
 * whose tensors are device pointers; `codec` is a device buffer of at least
 * bsq_codec_bytes, 256-byte aligned. Asynchronous on `stream`. */
bsq_status bsq_codec_bytes(const bsq_config *cfg, size_t *bytes);
bsq_status bsq_codec_prepare(const bsq_config *cfg, const bsq_decoder *dec,
                             void *codec, size_t codec_bytes, void *stream);

/* Encode n_mats matrices of one shape (Sections III-C to III-E):
 * protected-column scores key_j = g_j^2 sum_i W_ij^2 (fp64, rows in order),
 * TopK with ties to the lower column, quantisation of those columns in the
 * protect_format (eq. protected_8bit_scatter; int8 or FP8), then
 * per chunk and stage: sign code, decoded vector D_s(code), least-squares fp16
 * gain over the unprotected positions, residual update (fmaf chains in element
 * order). The outputs are bit-identical to the definition.
 *   W      device, bf16 or fp32, [n_mats][d_out][d_in] row-major, 16-byte aligned
 *   g      device fp32 [n_mats][d_in] activation statistic, or NULL for ones
 *          (protect_axis = 1: the rows are scored instead, key_i = g_i^2
 *          sum_j W_ij^2 with columns in order and g [n_mats][d_out]; the
 *          protected rows are then encoded as by bsq_encode_with_set)
 *   out    host struct of device output buffers sized by bsq_layer_sizes
 *          (times n_mats); out->d_out/d_in/pitch/k/n_mats must match
 *   err    device int32 error word; the caller zeroes it before the call; the
 *          library ORs BSQ_DEVERR_NONFINITE into it when W holds NaN or Inf
 *   ws     device workspace of bsq_workspace_bytes(ENCODE) bytes, 256-aligned */
bsq_status bsq_encode(const bsq_config *cfg, const void *codec, const void *W, int32_t w_dtype,
                      int64_t n_mats, int64_t d_out, int64_t d_in, const float *g,
                      const bsq_layer *out, int32_t *err, void *ws, size_t ws_bytes,
                      void *stream);

/* Encode with a given protected set (no selection): as bsq_encode, except that
 * the k slices on cfg->protect_axis are idx (device int32 [n_mats][k], each
 * matrix's entries strictly ascending and in [0, n) for the axis length n;
 * it may alias out->prot_idx). Column axis: quantisation (protect_format) of those
 * columns and BSQ on the rest of every row. Row axis: quantisation of
 * those rows (one scale per row, the absmax over the row / the format max); BSQ on the
 * other rows with no position masked; the protected rows get code 0 and gain
 * +0. An invalid set ORs BSQ_DEVERR_BAD_SET into *err (and the outputs are
 * unspecified); NaN or Inf in W ORs BSQ_DEVERR_NONFINITE. This is how the coupled set of bsq_coupled_select is
 * applied to the gate and up rows (axis 1) and the down columns (axis 0).
 * `g` is not used. Other arguments as for bsq_encode. With protect_axis = 1
 * and k > 0: d_out <= 2^18 and n_mats <= 65535 (BSQ_ERR_UNSUPPORTED beyond;
 * the same holds for bsq_encode on that axis). */
bsq_status bsq_encode_with_set(const bsq_config *cfg, const void *codec, const void *W, int32_t w_dtype,
                               int64_t n_mats, int64_t d_out, int64_t d_in, const int32_t *idx,
                               const bsq_layer *out, int32_t *err, void *ws, size_t ws_bytes,
                               void *stream);

/* Coupled MLP intermediate-channel selection (eq. mlp_coupled_protection):
 * for channel j < d_ffn,
 *   S_j = |g_gate_j| ||W_gate[j, :]|| + |g_up_j| ||W_up[j, :]|| + |g_down_j| ||W_down[:, j]||
 * with each squared norm an fp64 sum in element order (columns for the gate
 * and up rows, rows for the down column), the norm its correctly rounded fp64
 * square root and the three terms added left to right; then the k =
 * ceil(rho * d_ffn) largest, ties to the lower channel, ascending. Results
 * are bit-identical to that definition.
 *   W_gate, W_up  device [d_ffn][d_model], W_down device [d_model][d_ffn],
 *                 all bf16 or all fp32 (w_dtype), 16-byte aligned
 *   g_*           device fp32 [d_ffn] activation statistics, or NULL for ones
 *                 (taken by magnitude)
 *   idx           device int32 [k] output
 *   scores        device fp64 [d_ffn] output of S, or NULL
 *   err           device int32 error word (caller zeroes it); ORs BSQ_DEVERR_NONFINITE on NaN
 *                 or Inf in a weight
 *   ws            device workspace of bsq_workspace_bytes(SELECT, 1, d_ffn,
 *                 d_model) bytes, 256-byte aligned
 * protect_axis is ignored. */
bsq_status bsq_coupled_select(const bsq_config *cfg, const void *W_gate, const void *W_up, const void *W_down,
                              int32_t w_dtype, int64_t d_model, int64_t d_ffn, const float *g_gate,
                              const float *g_up, const float *g_down, int32_t *idx, double *scores,
                              int32_t *err, void *ws, size_t ws_bytes, void *stream);

/* Decode (eq. parallel_stage_decode, eq. protected_8bit_scatter):
 * W_hat[i][j] = sum_s gain_s * D_s(code_s)[j] as an fmaf chain over the stages
 * in fp32, then W_hat[:, idx_p] = q8[:, p] * scale_p (protect_axis = 1:
 * W_hat[idx_p, :] = q8[p, :] * scale_p). Bit-identical to the
 * definition for BSQ_F32 output; BSQ_BF16 rounds that value to nearest even.
 *   W_hat  device [n_mats][d_out][d_in] of out_dtype, 16-byte aligned */
bsq_status bsq_decode(const bsq_config *cfg, const void *codec, const bsq_layer *layer,
                      void *W_hat, int32_t out_dtype, void *stream);

/* One residual stage of a sequential decode, fp32 output (the stage-by-stage
 * form that eq. parallel_stage_decode replaces with one stage-parallel pass;
 * Section III-G compares the two as engineering cost):
 *   W_hat[i][j] = fmaf(gain_s, D_s(code_s)[j], accumulate ? W_hat[i][j] : 0)
 * over the unprotected positions of stage `stage` (0 <= stage < stages); the
 * call for the last stage then writes the protected columns (or rows) from
 * the protected payload. Calling it for stage = 0 .. stages-1, with accumulate = 0
 * then 1, leaves in W_hat the bits bsq_decode writes with BSQ_F32 output, at
 * the cost of one launch and one fp32 read-modify-write of W_hat per stage.
 *   W_hat  device fp32 [n_mats][d_out][d_in], 16-byte aligned */
bsq_status bsq_decode_stage(const bsq_config *cfg, const void *codec, const bsq_layer *layer,
                            int32_t stage, int32_t accumulate, void *W_hat, void *stream);

/* Fused decode-GEMV for a group of n matrices that read the same x (for
 * example q/k/v or gate/up), batch 1, without forming W_hat:
 *   y_g = W_hat_g x + B_g (A_g x)    for g = 0 .. n-1
 * computed as sum_c sum_s gain * <D_s(code), x~_c> + sum_p q8_p s_p x_{idx_p}
 * + B (A x), where x~ is x with the protected positions zeroed (Section V
 * names this direct computation from the codes as future work; the stage sum
 * is eq. parallel_stage_decode, the protected term eq. protected_8bit_scatter,
 * the LoRA term Section III-F).
 *   codecs  host array [n] of prepared codec device pointers (one per category)
 *   layers  host array [n]; all share d_in (and cfg); n_mats must be 1
 *   loras   host array [n] or NULL; an entry with rank 0 means no LoRA
 *   x       device [d_in], bf16 (16-byte aligned) or fp32 (x_dtype)
 *   y       host array [n] of device outputs [d_out_g], y_dtype (bf16 or fp32)
 *   ws      device workspace of bsq_workspace_bytes(GEMV, n, max d_out, d_in),
 *           256-byte aligned, ZERO-FILLED before its first use: a 256-byte
 *           header (its first word is the poison word), the LoRA vectors
 *           A_g x, the folded activations of the d = 16 symmetric decoder
 *           (see bsq_gemv_prepare) and flagged per-row partial sums that
 *           every call leaves at zero again. A workspace serves calls of one
 *           configuration and one d_in (any group size and d_out it was sized
 *           for); calls that share a workspace must not overlap.
 *   err     device int32 error word or NULL: TIMEOUT and POISONED (see
 *           BSQ_DEVERR_*) are ORed into it; without it those conditions
 *           still give NaN outputs and a poisoned workspace
 * bf16 x uses bf16 decoded values with fp32 accumulation; fp32 x uses the
 * fp32 decoder table and fp32 arithmetic throughout, and so does every
 * configuration with b != d (one wave per row over the 2^b-entry fp32
 * table; bsq_gemm likewise, with fp32 FMA over LDS tiles of decoded
 * weights instead of MFMA). With protect_axis = 1
 * the coded rows come from the streaming kernels and each protected row is
 * written afterwards as scale_p <q8[p, :], x> + B[row] (A x), one wave per
 * row (same stream).
 * bsq_gemv = bsq_gemv_prepare followed by bsq_gemv_run on the same stream. */
bsq_status bsq_gemv(const bsq_config *cfg, int32_t n, const void *const *codecs,
                    const bsq_layer *layers, const bsq_lora *loras,
                    const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                    void *ws, size_t ws_bytes, int32_t *err, void *stream);

/* bsq_gemv for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc. The
 * workspace is not an argument: the library keeps one zero-initialised
 * device array of BSQ_GEMV_NOALLOC_SCRATCH_BYTES (8 MiB) per GPU, held until
 * the process ends, and the call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine). Arguments, results and errors as bsq_gemv.
 *   clear_scratch  1: zero-fill the array (a kernel on `stream`) before the
 *                  product; needed only after a call reported
 *                  BSQ_DEVERR_TIMEOUT or BSQ_DEVERR_POISONED (synchronise
 *                  first). The first call on a GPU does this by itself.
 * BSQ_ERR_BUFFER_TOO_SMALL when the group's bsq_workspace_bytes(GEMV, ...)
 * exceeds the array (e.g. 2 x 25600 x 5120 at d = 8 needs 3.8 MiB). Every call
 * on a GPU shares that GPU's array, which keeps the last call's contents:
 * calls that overlap on one GPU (other streams, other host threads) race. */
bsq_status bsq_gemv_noalloc(const bsq_config *cfg, int32_t n, const void *const *codecs,
                            const bsq_layer *layers, const bsq_lora *loras,
                            const void *x, int32_t x_dtype, void *const *y, int32_t y_dtype,
                            int32_t clear_scratch, int32_t *err, void *stream);

/* Activation preparation of the GEMV: work that needs a reduction over all
 * of x, written into `ws` (one launch):
 *  - the LoRA vectors t_g = A_g x (fp32, 16 per member), for the paths that
 *    do not compute them inside bsq_gemv_run (that is, fp32 x, and d = 16
 *    with a decoder other than the width-16 symmetric one);
 *  - for the symmetric decoder at d = 16 with hidden width 16 and bf16 x, the
 *    decoder's output layer folded into the masked activations: per member,
 *    stage and chunk c, u = W2^T x~_c and b2 . x~_c (so that
 *    <D(code), x~_c> = <relu(W1 q + b1), u> + b2 . x~_c), u stored in fp16
 *    with a power-of-two scale.
 * Launches nothing when neither applies. Arguments as for bsq_gemv; `codecs`
 * may be NULL unless the folded activations are needed. (Masking x for the
 * other configurations and scaling the protected activations happen inside
 * bsq_gemv_run.) */
bsq_status bsq_gemv_prepare(const bsq_config *cfg, int32_t n, const void *const *codecs,
                            const bsq_layer *layers, const bsq_lora *loras, const void *x,
                            int32_t x_dtype, void *ws, size_t ws_bytes, void *stream);

/* The streaming product of the GEMV, alone: reads x, the code and gain
 * planes, the protected payload and LoRA A and B once, and whatever a preceding
 * bsq_gemv_prepare (same group, same x) left in `ws` on the same stream.
 * With bf16 x at d = 8 (and d = 16 with the width-16 symmetric decoder) the
 * LoRA vectors are computed inside this launch. Limits of the bf16 path:
 * d_in <= 65536 and k <= 4096. `err` as for bsq_gemv. */
bsq_status bsq_gemv_run(const bsq_config *cfg, int32_t n, const void *const *codecs,
                        const bsq_layer *layers, const bsq_lora *loras, const void *x,
                        int32_t x_dtype, void *const *y, int32_t y_dtype, void *ws,
                        size_t ws_bytes, int32_t *err, void *stream);

/* Fused decode-GEMM for M tokens, Y = X W_hat^T + (X A^T) B^T: the batched
 * form of the product bsq_gemv computes (the direct computation from the
 * binary codes that Section V names as future work; stage sum of
 * eq. parallel_stage_decode, protected term of eq. protected_8bit_scatter,
 * LoRA term of Section III-F). Each lane decodes its weight fragments from
 * the code and gain planes straight into bf16 MFMA operands (fp16 decoder
 * tables in LDS, fp32 fma over the stages), so W_hat is never formed:
 *   X  device bf16 [M][ldx] (ldx >= d_in, multiple of 8)
 *   Y  device [M][ldy] of y_dtype (bf16 or fp32), ldy >= d_out
 *   ws device workspace of bsq_workspace_bytes(GEMM, 1, d_out, d_in, M),
 *      256-byte aligned, any contents: a 256-byte header the call leaves
 *      untouched, then scratch (X with the protected columns zeroed, the
 *      gathered protected activations, X A^T, split-K partials). One
 *      workspace serves GEMM calls of any shape; calls that share it must
 *      not overlap.
 *   err device int32 error word or NULL (accepted for symmetry with
 *      bsq_gemv; no workgroup of the product waits for another, so nothing
 *      is reported).
 * The K steps of a tile may be split over several blocks; their fp32
 * partials are summed in a fixed order by a second launch on the same
 * stream, so results are deterministic. With
 * protect_axis = 1 each protected row's column of Y is written afterwards as
 * scale_p X q8[p, :]^T + (X A^T) B[row]^T (same stream); that pass takes four
 * tokens per block, so M <= 262140 there (BSQ_ERR_UNSUPPORTED beyond). */
bsq_status bsq_gemm(const bsq_config *cfg, const void *codec, const bsq_layer *layer,
                    const bsq_lora *lora, const void *X, int32_t x_dtype, int64_t M,
                    int64_t ldx, void *Y, int32_t y_dtype, int64_t ldy,
                    void *ws, size_t ws_bytes, int32_t *err, void *stream);

/* ------------------------------------------------------------------------
 * Codec training (Section III-C; eq. codec_loss, eq. codec_loss_terms;
 * Section III-G, category-batched codec optimisation).
 *
 * One stage codec with the LINEAR encoder and the symmetric decoder without
 * residual block (cfg->encoder = BSQ_ENC_LINEAR, cfg->dec_kind = BSQ_DEC_MLP,
 * d and b 8 or 16, h = cfg->hidden) is trained on weight chunks: for a
 * mini-batch of N chunks x_i,
 *   z = E x, u = z / ||z||, q = sign(u) / sqrt(b), x_hat = D(q) with the
 *   straight-through estimator (the decoder reads q; the gradient reaching q
 *   is passed to u; a chunk with z = 0 has u = 0 and passes none),
 *   L_rec = 1/N sum ||x_hat - x||^2,  L_com = 1/N sum ||u - sg(q)||^2,
 *   p_ij = [sigma(-t_ij), sigma(t_ij)], t_ij = 2 tau u_ij / sqrt(b),
 *   L_ent = 1/N sum_i sum_j H(p_ij) - gamma sum_j H(mean_i p_ij),
 *   L = L_rec + lambda_c L_com + lambda_e L_ent   (natural logarithms).
 * The parameters are one fp32 vector theta, laid out
 *   E [b][d] | W1 [h][b] | b1 [h] | W2 [d][h] | b2 [d]
 * (bsq_train_param_count floats; the first b d and the decoder part are what
 * bsq_codec_prepare takes as E, W1, b1, W2, b2). The code bits of z and the
 * ReLU mask of the hidden layer are decided in fp32 by the same fmaf chains
 * as the encoder's; every reduction runs in a fixed order, so a step is
 * deterministic.
 * ------------------------------------------------------------------------ */
typedef struct {
    float lambda_c;  /* commitment weight */
    float lambda_e;  /* entropy weight */
    float gamma;     /* batch-entropy weight */
    float tau;       /* bit-probability temperature */
    float lr, beta1, beta2, eps;  /* Adam (Kingma & Ba 2015) */
} bsq_train_hparams;

bsq_status bsq_train_param_count(const bsq_config *cfg, int64_t *count);
/* device workspace for a mini-batch of n chunks (256-byte aligned) */
bsq_status bsq_train_workspace_bytes(const bsq_config *cfg, int64_t n, size_t *bytes);

/* Loss and gradient of one mini-batch.
 *   chunks   device [n_total][d], fp32 or bf16 (x_dtype): the chunks of a
 *            category, e.g. its stacked layers [n_mats][d_out][d_in] viewed
 *            as n_mats d_out d_in / d chunks (row-major chunks are contiguous)
 *   idx      device int64 [n] chunk indices of the mini-batch, or NULL for
 *            chunks 0 .. n-1; an index outside [0, n_total) ORs
 *            BSQ_DEVERR_BAD_SET into *err and reads chunk 0
 *   theta    device fp32 [P] (read)
 *   grad     device fp32 [P] (written): dL/dtheta
 *   loss     device fp32 [4] (written): L, L_rec, L_com, L_ent
 *   err      device int32 error word or NULL
 *   ws       device workspace of bsq_train_workspace_bytes(cfg, n) */
bsq_status bsq_train_grad(const bsq_config *cfg, const bsq_train_hparams *hp, const void *chunks, int32_t x_dtype,
                          int64_t n_total, const int64_t *idx, int64_t n, const float *theta, float *grad,
                          float *loss, int32_t *err, void *ws, size_t ws_bytes, void *stream);

/* One Adam step in place, bias-corrected, step = 1, 2, ...:
 *   m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 *   theta -= lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * theta, m, v device fp32 [P] (m, v zero before step 1); grad as written by
 * bsq_train_grad. */
bsq_status bsq_train_adam(const bsq_config *cfg, const bsq_train_hparams *hp, int32_t step, float *theta,
                          const float *grad, float *m, float *v, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* BSQ_H */
