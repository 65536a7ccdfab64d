// Fused decode-GEMV at batch 1 (the direct computation from binary spherical
// codes that Section V names as future work):
//   y_i = sum_c sum_s gain_s(i,c) * <D_s(code_s(i,c)), x~_c>
//         + sum_p q8(i,p) * (scale_p x_{idx_p}) + sum_r B(i,r) (A x)_r
// where x~ is x with the protected input columns zeroed (those columns come
// from the int8 path, eq. protected_8bit_scatter) and the stage sum is the
// parallel residual decoding of eq. parallel_stage_decode.
//
// Kernels:
//  * gemv_prep_kernel (bsq_gemv_prepare): the d = 16 symmetric decoder's
//    folded activation records (the output layer folded into x~ per chunk),
//    and the LoRA vectors A x for the kernels that do not compute them.
//  * gemv_lane_kernel (bf16 activations, d = 8, and d = 16 with the
//    symmetric decoder of hidden width 16): a lane owns a row of a 64-row
//    tile, the tile's activations are wave-uniform scalar operands, the
//    decoder comes from LDS tables; extra workgroups ahead of the tiles
//    compute the LoRA vectors A x. The headline kernel.
//  * gemv_stream_kernel (bf16 activations, other d = 16 decoders): a thread
//    owns a 128-input segment of x~ and walks down rows, table lookups from
//    global memory.
//  * gemv_f32_kernel (fp32 activations): one wave per row, fp32 tables.
#include <mutex>

#include "bsq_internal.h"

namespace bsq {
namespace {

// Workspace: a 256-byte header (its first word is the poison word, nonzero
// once a call gave up waiting for a partial result and left flagged slots
// behind), the LoRA vectors of up to BSQ_MAX_GROUP members, then the flagged
// partial slots. The slots start at the same offset for every group size, so
// a workspace shared by groups of different sizes keeps its slots at zero
// between calls.
constexpr size_t GEMV_HDR = 256;
// bsq_gemv_noalloc's scratch array: the folded activation records of the
// d = 16 symmetric decoder in its last 2 MiB, everything else from the front
constexpr size_t GEMV_SCRATCH_XP_BYTES = size_t(2) << 20;
constexpr size_t gemv_t_bytes() { return (size_t(BSQ_MAX_GROUP) * BSQ_MAX_LORA_RANK * 4 + 255) & ~size_t(255); }

// The d = 16 symmetric decoder path (hidden width 16) evaluates the decoder
// from split pre-activation tables and folded activations.
inline bool gemv_split16(const bsq_config &cfg) { return codec_has_split(cfg) && cfg.hidden == 16; }

// Workspace of that path: a 64-byte folded-activation record per (member,
// stage, chunk), for BSQ_MAX_GROUP members so that the slots behind it start
// at the same offset for every group size of one configuration and d_in.
inline bool gemv_lane_path(const bsq_config &cfg, int x_dtype)
{
    return x_dtype == BSQ_BF16 && cfg.b == cfg.d && (cfg.d == 8 || gemv_split16(cfg));
}

inline size_t gemv_xp_bytes(const bsq_config &cfg, int64_t pitch)
{
    return gemv_split16(cfg) ? size_t(BSQ_MAX_GROUP) * cfg.stages * size_t(pitch) * 64 : 0;
}

// row-lane kernel: largest padded int8 row that a finishing slice brings to
// LDS (64 rows x 256 B = 16 KiB); longer rows are read from global memory
constexpr int64_t LANE_Q8_LDS_MAX = 256;


typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}


__device__ __forceinline__ float half_lo(uint32_t w) { return f16_bits_to_f32(uint16_t(w & 0xffffu)); }
__device__ __forceinline__ float half_hi(uint32_t w) { return f16_bits_to_f32(uint16_t(w >> 16)); }

__device__ __forceinline__ bool is_protected(const int32_t *idx, int64_t k, int64_t j)
{
    int64_t lo = 0, hi = k;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (idx[mid] < j) lo = mid + 1;
        else hi = mid;
    }
    return lo < k && idx[lo] == j;
}

struct GemvMat {
    const void *codes[BSQ_MAX_STAGES];
    const uint16_t *gains[BSQ_MAX_STAGES];
    const uint16_t *tab16[BSQ_MAX_STAGES];
    const float *tab32[BSQ_MAX_STAGES];
    const int32_t *idx;
    const int8_t *q8;
    const float *scale;
    const uint16_t *A;  // LoRA A [rank][d_in], bf16
    const uint16_t *B;  // LoRA B [d_out][rank], bf16
    int rank;
    const uint32_t *bits;  // protected-column bitmap [pitch * d / 32]
    // d = 16 symmetric decoder: split pre-activation tables (fp16 [2][2][256][8])
    // and the fp32 W2 [16][16], b2 [16] of each stage
    const uint16_t *split[BSQ_MAX_STAGES];
    const float *w2[BSQ_MAX_STAGES];
    const float *b2[BSQ_MAX_STAGES];
    uint32_t *xp;  // workspace: folded activation records [S][pitch][16] (d = 16 decoder path)
    int64_t d_out;
    int64_t block_begin;  // first block of this member in the grid
    int64_t rg_begin;     // row-lane kernel: first 64-row group of this member (partial-sum slots)
    int64_t lora_begin;   // row-lane kernel: first LoRA workgroup of this member (one per rank index)
    float *t;             // workspace: A x, [16]
    void *y;
};

struct GemvArgs {
    // first block of each member in the row-lane kernel's tile grid (INT32_MAX
    // past the last member), the LoRA workgroups ahead of them, and the tile
    // counts: what every workgroup reads first, together, at the front of the
    // arguments (one batch of scalar loads before the member's own fields)
    int32_t bb[BSQ_MAX_GROUP];
    int32_t lora_blocks32;
    int n, stages;
    int64_t d_in, pitch, k, nseg, rs, rpb;
    int64_t nblk, q;   // row-lane kernel: 16-chunk blocks per row, slices per 64-row group
    uint64_t *slots;   // row-lane kernel: {flag, partial} [row groups][q - 1][64], zero between calls
    uint64_t *tslots;  // row-lane kernel: {flag, (A x)_r} [row groups][16], zero between calls
    int64_t lora_blocks;  // row-lane kernel: LoRA workgroups ahead of the tiles' workgroups
    const void *x;
    int x_bf16, y_bf16;
    uint32_t *poison;  // row-lane kernel: the workspace's poison word
    int32_t *err;      // caller's device error word, or null
    int spin_limit;    // polls before a wait gives up (wait_limit())
    int pfmt;          // bsq_prot_format of the protected payload
    GemvMat mat[BSQ_MAX_GROUP];
};

__device__ __forceinline__ float load_x(const void *x, int64_t j, int bf)
{
    return bf ? bf16_to_f32(static_cast<const uint16_t *>(x)[j]) : static_cast<const float *>(x)[j];
}

// ---------------------------------------------------------------------------
// Activation prep, one launch:
//  * blocks [0, n * 16): the LoRA vectors t[m][r] = sum_j A[r][j] x_j
//    (unmasked x), one block per (member, rank index);
//  * the rest (d = 16 symmetric decoder only): one block per (member,
//    stage, 16 chunks), sixteen threads per chunk c, fold the decoder's
//    output layer into the masked activations of the chunk:
//    u_k = sum_i W2[i][k] x~_{16c+i} and beta = sum_i b2[i] x~_{16c+i}, so
//    that <D(code), x~_c> = <relu(a), u> + beta with a the hidden
//    pre-activation of the code. The record is u in fp16 scaled by 2^-e (e
//    puts max |u| in [2^13, 2^14), so no u overflows or loses range), then
//    beta 2^-e and 2^e as fp32, in a 64-byte slot. Chunks past the row
//    (pitch padding) get zeros.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemv_prep_kernel(const GemvArgs a, int lora_blocks)
{
    __shared__ float red[256];
    const int t = threadIdx.x;
    if (int(blockIdx.x) < lora_blocks) {
        const int m = blockIdx.x / BSQ_MAX_LORA_RANK;
        const int r = blockIdx.x % BSQ_MAX_LORA_RANK;
        const GemvMat &M = a.mat[m];
        if (r >= M.rank) return;
        float acc = 0.0f;
        for (int64_t j = t; j < a.d_in; j += 256)
            acc = __builtin_fmaf(bf16_to_f32(M.A[int64_t(r) * a.d_in + j]), load_x(a.x, j, a.x_bf16), acc);
        red[t] = acc;
        __syncthreads();
        for (int o = 128; o > 0; o >>= 1) {
            if (t < o) red[t] += red[t + o];
            __syncthreads();
        }
        if (t == 0) M.t[r] = red[0];
        return;
    }
    // folded activations: one block per (member, stage, 16-chunk block),
    // thread t = 16 (chunk in the block) + hidden unit k
    __shared__ float s_w2[256], s_b2[16], s_x[16][17];
    const int64_t bid = int64_t(blockIdx.x) - lora_blocks;
    const int64_t nblk = a.pitch / 16;
    const int m = int(bid / (int64_t(a.stages) * nblk));
    if (m >= a.n) return;
    const int s = int((bid / nblk) % a.stages);
    const int64_t c = (bid % nblk) * 16 + t / 16;
    const int k = t & 15;
    const GemvMat &M = a.mat[m];
    s_w2[t] = M.w2[s][t];  // W2 [i][k], i the output element
    if (t < 16) s_b2[t] = M.b2[s][t];
    {
        const int64_t col = 16 * c + k;  // this thread's element of the chunk
        float v = (col < a.d_in) ? load_x(a.x, col, a.x_bf16) : 0.0f;
        if (a.k > 0 && col < a.d_in && ((M.bits[col >> 5] >> (col & 31)) & 1u)) v = 0.0f;
        s_x[t / 16][k] = v;
    }
    __syncthreads();
    const float *xc = s_x[t / 16];
    float u = 0.0f, beta = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        u = __builtin_fmaf(s_w2[i * 16 + k], xc[i], u);
        beta = __builtin_fmaf(s_b2[i], xc[i], beta);
    }
    float amax = __builtin_fabsf(u);
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) amax = __builtin_fmaxf(amax, __shfl_xor(amax, o, 16));
    int e = 0;
    if (amax > 0.0f && amax <= 3.0e38f) {
        int ex;
        __builtin_frexpf(amax, &ex);  // amax = f 2^ex, f in [0.5, 1)
        e = ex - 14;
        e = (e < -110) ? -110 : (e > 110 ? 110 : e);
    }
    uint32_t *rec = M.xp + (int64_t(s) * a.pitch + c) * 16;
    reinterpret_cast<uint16_t *>(rec)[k] = __builtin_bit_cast(uint16_t, static_cast<_Float16>(__builtin_ldexpf(u, -e)));
    if (k == 0) {
        rec[8] = __float_as_uint(__builtin_ldexpf(beta, -e));
        rec[9] = __float_as_uint(__builtin_ldexpf(1.0f, e));
    }
}

// ---------------------------------------------------------------------------
// Streaming kernel, bf16 activations.
// ---------------------------------------------------------------------------
template <int D, int S>
struct RowData {
    uint4 c[S];
    uint4 g[S][D == 8 ? 2 : 1];
};

template <int D, int S>
__device__ __forceinline__ void load_row(RowData<D, S> &r, const GemvMat &M, int64_t off)
{
#pragma unroll
    for (int s = 0; s < S; ++s) {
        if constexpr (D == 8)
            r.c[s] = *reinterpret_cast<const uint4 *>(static_cast<const uint8_t *>(M.codes[s]) + off);
        else
            r.c[s] = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(M.codes[s]) + off);
        const uint4 *gp = reinterpret_cast<const uint4 *>(M.gains[s] + off);
        r.g[s][0] = gp[0];
        if constexpr (D == 8) r.g[s][1] = gp[1];
    }
}

template <int D, int S>
__device__ __forceinline__ float row_dot(const RowData<D, S> &r, const uint4 (&xv)[16], const uint4 *s_tab,
                                         const GemvMat &M)
{
    constexpr int SEGC = 128 / D;
    float acc = 0.0f;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint32_t *cws = reinterpret_cast<const uint32_t *>(&r.c[s]);
        const uint32_t *gws = reinterpret_cast<const uint32_t *>(&r.g[s][0]);
#pragma unroll
        for (int kk = 0; kk < SEGC; ++kk) {
            float dsum;
            if constexpr (D == 8) {
                const uint32_t code = (cws[kk >> 2] >> (8 * (kk & 3))) & 0xffu;
                const uint4 e = s_tab[s * 256 + code];
                const uint4 x = xv[kk];
                dsum = dot2_bf16(e.x, x.x, 0.0f);
                dsum = dot2_bf16(e.y, x.y, dsum);
                dsum = dot2_bf16(e.z, x.z, dsum);
                dsum = dot2_bf16(e.w, x.w, dsum);
            } else {
                const uint32_t code = (cws[kk >> 1] >> (16 * (kk & 1))) & 0xffffu;
                const uint4 *ep = reinterpret_cast<const uint4 *>(M.tab16[s]) + size_t(code) * 2;
                const uint4 e0 = ep[0], e1 = ep[1];
                const uint4 x0 = xv[2 * kk], x1 = xv[2 * kk + 1];
                dsum = dot2_bf16(e0.x, x0.x, 0.0f);
                dsum = dot2_bf16(e0.y, x0.y, dsum);
                dsum = dot2_bf16(e0.z, x0.z, dsum);
                dsum = dot2_bf16(e0.w, x0.w, dsum);
                dsum = dot2_bf16(e1.x, x1.x, dsum);
                dsum = dot2_bf16(e1.y, x1.y, dsum);
                dsum = dot2_bf16(e1.z, x1.z, dsum);
                dsum = dot2_bf16(e1.w, x1.w, dsum);
            }
            const uint32_t gword = gws[kk >> 1];
            const float g = (kk & 1) ? half_hi(gword) : half_lo(gword);
            acc = __builtin_fmaf(g, dsum, acc);
        }
    }
    return acc;
}

template <int D, int S>
__global__ __launch_bounds__(512) void gemv_stream_kernel(const GemvArgs a)
{
    extern __shared__ uint4 s_mem[];
    const int NT = blockDim.x;
    const int t = threadIdx.x;
    const int nseg = int(a.nseg), rs = int(a.rs), rpb = int(a.rpb);
    const int64_t words = (a.d_in + 31) / 32;
    // LDS: [tables (d = 8)] [partials rpb x nseg] [bitmap words] [xs k]
    uint4 *s_tab = s_mem;
    float *s_red = reinterpret_cast<float *>(s_mem + ((D == 8) ? S * 256 : 0));
    uint32_t *s_bits = reinterpret_cast<uint32_t *>(s_red + rpb * nseg);
    float *s_xs = reinterpret_cast<float *>(s_bits + ((words + 3) & ~int64_t(3)));

    int m = 0;
    while (m + 1 < a.n && int64_t(blockIdx.x) >= a.mat[m + 1].block_begin) ++m;
    const GemvMat &M = a.mat[m];
    const int64_t row_begin = (int64_t(blockIdx.x) - M.block_begin) * rpb;
    const int nrows = int((M.d_out - row_begin < rpb) ? (M.d_out - row_begin) : rpb);
    const int slot = t / nseg, seg = t - slot * nseg;
    const bool active = slot < rs;
    constexpr int SEGC = 128 / D;

    // issue this thread's first HBM loads before the block setup: its x
    // segment and its first two rows (rows i = slot, slot + rs, ...)
    uint4 xv[16];
    RowData<D, S> r0, r1;
    const int64_t j0 = int64_t(seg) * 128;
    const int nmine = (active && nrows > slot) ? (nrows - slot + rs - 1) / rs : 0;
    static_assert(SEGC == 8, "the streaming kernel reads one 8-chunk tile block per segment");
    const int64_t row0 = row_begin + slot;
    const int64_t base = tile_index(row0, int64_t(seg) * SEGC, a.pitch);
    if (active) {
        const uint4 *xp = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(a.x) + j0);
#pragma unroll
        for (int q = 0; q < 16; ++q) xv[q] = (j0 + 8 * q < a.d_in) ? xp[q] : make_uint4(0, 0, 0, 0);
        if (nmine > 0) load_row<D, S>(r0, M, base);
        if (nmine > 1) load_row<D, S>(r1, M, tile_index(row0 + rs, int64_t(seg) * SEGC, a.pitch));
    }

    // block setup while the loads are in flight: decoder table, protected
    // bitmap, scaled protected activations
    if constexpr (D == 8) {
        for (int e = t; e < S * 256; e += NT) s_tab[e] = reinterpret_cast<const uint4 *>(M.tab16[e >> 8])[e & 255];
    }
    if (a.k > 0) {
        for (int64_t w = t; w < words; w += NT) s_bits[w] = 0u;
        __syncthreads();
        for (int64_t p = t; p < a.k; p += NT) {
            const int32_t j = M.idx[p];
            if (j >= 0 && j < a.d_in) {
                atomicOr(&s_bits[j >> 5], 1u << (j & 31));
                s_xs[p] = M.scale[p] * load_x(a.x, j, 1);
            } else {
                s_xs[p] = 0.0f;
            }
        }
    }
    __syncthreads();

    if (active) {
        if (a.k > 0) {
#pragma unroll
            for (int wq = 0; wq < 4; ++wq) {
                const int64_t w = (j0 >> 5) + wq;
                const uint32_t bits = (w < words) ? s_bits[w] : 0u;
                if (bits) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        uint32_t *xw = reinterpret_cast<uint32_t *>(&xv[wq * 4 + q]);
#pragma unroll
                        for (int h = 0; h < 4; ++h) {
                            const uint32_t b2 = bits >> (8 * q + 2 * h);
                            const uint32_t keep = ((b2 & 1u) ? 0u : 0x0000ffffu) | ((b2 & 2u) ? 0u : 0xffff0000u);
                            xw[h] &= keep;
                        }
                    }
                }
            }
        }
        // two rows in flight: compute one while the next but one loads
        int i = 0;
        for (; i + 1 < nmine; i += 2) {
            s_red[(slot + i * rs) * nseg + seg] = row_dot<D, S>(r0, xv, s_tab, M);
            if (i + 2 < nmine) load_row<D, S>(r0, M, tile_index(row0 + int64_t(i + 2) * rs, int64_t(seg) * SEGC, a.pitch));
            s_red[(slot + (i + 1) * rs) * nseg + seg] = row_dot<D, S>(r1, xv, s_tab, M);
            if (i + 3 < nmine) load_row<D, S>(r1, M, tile_index(row0 + int64_t(i + 3) * rs, int64_t(seg) * SEGC, a.pitch));
        }
        if (i < nmine) s_red[(slot + i * rs) * nseg + seg] = row_dot<D, S>(r0, xv, s_tab, M);
    }
    __syncthreads();

    // reduce the segment partials of each row and add the int8 and LoRA terms
    int G = 64;
    while (G > 1 && G * nrows > NT) G >>= 1;
    const int g = t & (G - 1);
    for (int r = t / G; r < nrows; r += NT / G) {
        const int64_t row = row_begin + r;
        float v = 0.0f;
        const float *rp = s_red + r * nseg;
        for (int q = g; q < nseg; q += G) v += rp[q];
        for (int64_t p = g; p < a.k; p += G)
            v = __builtin_fmaf(payload_to_f32(uint8_t(M.q8[row * q8_pitch(a.k) + p]), a.pfmt), s_xs[p], v);
        for (int q = g; q < M.rank; q += G) v = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], v);
        for (int o = G >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        if (g == 0) {
            if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(v);
            else static_cast<float *>(M.y)[row] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// Row-lane kernel (d = 8, bf16 activations).
//
// Tile = 64 rows x 16 chunks (128 inputs), stored contiguously (1 KiB of codes
// and 2 KiB of gains per stage); the tiles of a 64-row group follow each other
// in memory. A lane owns one row, so the 128-input activation block of a tile
// is wave-uniform: it is read with scalar loads, masked in scalar registers
// with the layer's protected-column bitmap, and is the scalar operand of
// v_dot2_f32_bf16. Table lookups come from LDS.
//
// The grid is many short workgroups rather than a persistent one: a workgroup
// of four waves owns one slice of 4 * TPW consecutive tiles of one row group,
// each wave streams its TPW tiles two at a time, and the four wave sums of a
// row are added in LDS in wave order. Short workgroups let the hardware
// dispatcher balance the load over the CUs as they free up.
//
// The Q slices of a row group are consecutive workgroups. Slices 0 .. Q-2
// each publish their 64 partial sums together with a ready flag (one 64-bit
// agent-scope atomic store per lane, so data and flag are seen together) and
// are done; the last slice adds the int8 and LoRA terms to its own sum
// (work that does not depend on the others, so it overlaps the wait), then
// polls those slots, adds them in slice order, then its own sum, clears the
// slots and stores.
// Workgroups are dispatched in index order, so the slices it waits for are
// running or done; a bounded poll turns a never-expected stall into NaN
// outputs instead of a hang. No counter, no cache-wide writeback or
// invalidate, and no contributor waits.
//
// The tile loop is branch-free around its loads: a conditional load makes
// the compiler wait for it at once, which would leave one tile in flight.
// ---------------------------------------------------------------------------
template <int D, int S>
struct LaneBlk {
    uint4 c[S][D / 8];  // 16 codes of the lane's row (one byte each at d = 8, two at d = 16)
    uint4 g[S][2];      // 16 fp16 gains
};

// The member's plane pointers, read from the kernel arguments once.
template <int S>
struct LanePlanes {
    const uint8_t *codes[S];
    const uint16_t *gains[S];
};

template <int D, int S>
__device__ __forceinline__ void lane_load(LaneBlk<D, S> &b, const LanePlanes<S> &P, int64_t off)
{
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint4 *cp = reinterpret_cast<const uint4 *>(P.codes[s] + off * (D / 8));
#pragma unroll
        for (int h = 0; h < D / 8; ++h) b.c[s][h] = cp[h];
        const uint4 *gp = reinterpret_cast<const uint4 *>(P.gains[s] + off);
        b.g[s][0] = gp[0];
        b.g[s][1] = gp[1];
    }
}

// The LoRA term (tv = A x) of one output row (row < d_out), added to acc.
// The rank-16 row of B is loaded unconditionally (indices clamped to the
// rank) so that its loads are in flight together.
__device__ __forceinline__ float lane_lora_term(const GemvMat &M, int64_t row, float acc,
                                                const float (&tv)[BSQ_MAX_LORA_RANK])
{
    if (M.rank > 0) {
        const uint16_t *br = M.B + row * M.rank;
        uint16_t bq[BSQ_MAX_LORA_RANK];
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) bq[q] = br[(q < M.rank) ? q : M.rank - 1];
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) {
            const float f = __builtin_fmaf(bf16_to_f32(bq[q]), tv[q], acc);
            acc = (q < M.rank) ? f : acc;
        }
    }
    return acc;
}

__device__ __forceinline__ void lane_store(const GemvArgs &a, const GemvMat &M, int64_t row, float v)
{
    if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(v);
    else static_cast<float *>(M.y)[row] = v;
}

// Sixteen protected columns of one row: stored bytes (one 16-byte word, in
// format FMT) against the scaled activations xs[0 .. 15] (LDS, 16-byte
// aligned, zero past k).
template <int FMT>
__device__ __forceinline__ float q8_block_t(uint4 qv, const float *xs, float acc)
{
    const float4 *x4 = reinterpret_cast<const float4 *>(xs);
    const float4 xa = x4[0], xb = x4[1], xc = x4[2], xd = x4[3];
    const float xv[16] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w,
                          xc.x, xc.y, xc.z, xc.w, xd.x, xd.y, xd.z, xd.w};
    const uint32_t qw[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        acc = __builtin_fmaf(payload_byte<FMT, 0>(qw[w]), xv[4 * w], acc);
        acc = __builtin_fmaf(payload_byte<FMT, 1>(qw[w]), xv[4 * w + 1], acc);
        acc = __builtin_fmaf(payload_byte<FMT, 2>(qw[w]), xv[4 * w + 2], acc);
        acc = __builtin_fmaf(payload_byte<FMT, 3>(qw[w]), xv[4 * w + 3], acc);
    }
    return acc;
}

// (the format dispatched once per sixteen columns, a uniform branch)
__device__ __forceinline__ float q8_block(uint4 qv, const float *xs, float acc, int fmt)
{
    if (fmt == BSQ_PROT_E4M3) return q8_block_t<BSQ_PROT_E4M3>(qv, xs, acc);
    if (fmt == BSQ_PROT_E5M2) return q8_block_t<BSQ_PROT_E5M2>(qv, xs, acc);
    return q8_block_t<BSQ_PROT_INT8>(qv, xs, acc);
}

// The protected columns of 16-column words w0, w0 + step, ... of one row
// (row < d_out) added to acc, the row's stored bytes read from global
// memory: four words at a time, all issued before any is used (indices
// clamped to the padded row, words past it zeroed), then one after the other.
__device__ __forceinline__ float lane_q8_global(const GemvArgs &a, const GemvMat &M, const float *s_xs, int64_t row,
                                                int64_t w0, int64_t step, float acc)
{
    const int64_t nw = q8_pitch(a.k) / 16;  // 16-byte words per row
    const uint4 *qr = reinterpret_cast<const uint4 *>(M.q8 + row * q8_pitch(a.k));
    for (int64_t w = w0; w < nw; w += 4 * step) {
        uint4 qv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) qv[u] = qr[(w + u * step < nw) ? w + u * step : nw - 1];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t wu = w + u * step;
            const uint4 q = (wu < nw) ? qv[u] : make_uint4(0, 0, 0, 0);
            acc = q8_block(q, s_xs + 16 * ((wu < nw) ? wu : nw - 1), acc, a.pfmt);
            asm volatile("" : "+v"(acc));  // one word's activations live at a time
        }
    }
    return acc;
}

// The protected columns of words w0, w0 + step, ... of one row (row <
// d_out), with the row's stored bytes in LDS (s_q8 [64][kp], this lane's row
// at (row % 64) kp) or else in global memory, added to acc in word order.
__device__ __forceinline__ float lane_q8_term(const GemvArgs &a, const GemvMat &M, const float *s_xs,
                                              const int8_t *s_q8, bool q8_lds, int64_t row, int64_t w0, int64_t step,
                                              float acc)
{
    if (a.k > 0) {
        if (q8_lds) {
            const int64_t nw = q8_pitch(a.k) / 16;
            const uint4 *qr = reinterpret_cast<const uint4 *>(s_q8 + (row & 63) * q8_pitch(a.k));
            int64_t w = w0;
            for (; w + step < nw; w += 2 * step) {  // two words per step, their LDS reads together
                const uint4 q0 = qr[w], q1 = qr[w + step];
                acc = q8_block(q0, s_xs + 16 * w, acc, a.pfmt);
                acc = q8_block(q1, s_xs + 16 * (w + step), acc, a.pfmt);
            }
            if (w < nw) acc = q8_block(qr[w], s_xs + 16 * w, acc, a.pfmt);
        } else {
            acc = lane_q8_global(a, M, s_xs, row, w0, step, acc);
        }
    }
    return acc;
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
typedef const u32x4 __attribute__((address_space(4))) *cx4_ptr;
typedef const u32x16 __attribute__((address_space(4))) *cx16_ptr;

// Zero the protected inputs of one 32-input group held in scalar registers
// (16 bf16 pairs); `bw` is the group's bitmap word, bit 2w (2w + 1) for the
// low (high) half of word w. Straight-line scalar code under one uniform
// branch: most groups hold no protected input.
__device__ __forceinline__ u32x16 mask_group(u32x16 v, uint32_t bw)
{
    if (bw) {
#pragma unroll
        for (int w = 0; w < 16; ++w) {
            const uint32_t lo = uint32_t(int32_t(bw << (31 - 2 * w)) >> 31);   // 0 or ~0
            const uint32_t hi = uint32_t(int32_t(bw << (30 - 2 * w)) >> 31);
            v[w] &= ~((lo & 0x0000ffffu) | (hi & 0xffff0000u));
        }
    }
    return v;
}

// One 32-input group (chunks 4z .. 4z+3 of a tile) of the lane's row, all
// stages: table entries from LDS, dotted with the wave-uniform activations.
template <int S>
__device__ __forceinline__ float lane_group(const LaneBlk<8, S> &b, int z, const u32x16 &xz, const uint4 *s_tab,
                                            float acc)
{
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint32_t cw = (z == 0) ? b.c[s][0].x : (z == 1) ? b.c[s][0].y : (z == 2) ? b.c[s][0].z : b.c[s][0].w;
        const uint4 gq = b.g[s][z >> 1];
        const uint32_t g0 = (z & 1) ? gq.z : gq.x;
        const uint32_t g1 = (z & 1) ? gq.w : gq.y;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            // byte offset of the code's 16-byte entry (one shift of the
            // selected byte; the stage's base is the instruction's offset)
            const uint32_t off = ((cw >> (8 * kk)) & 0xffu) << 4;
            const uint4 e = *reinterpret_cast<const uint4 *>(reinterpret_cast<const char *>(s_tab + s * 256) + off);
            float dsum = dot2_bf16(e.x, xz[4 * kk + 0], 0.0f);
            dsum = dot2_bf16(e.y, xz[4 * kk + 1], dsum);
            dsum = dot2_bf16(e.z, xz[4 * kk + 2], dsum);
            dsum = dot2_bf16(e.w, xz[4 * kk + 3], dsum);
            const uint32_t gw = (kk < 2) ? g0 : g1;
            const float g = (kk & 1) ? half_hi(gw) : half_lo(gw);
            acc = __builtin_fmaf(g, dsum, acc);
        }
    }
    return acc;
}

// One full tile (128 inputs of block b): four groups of 32 activations, each
// read with one scalar load (xb: the tile's activations, 4 groups) and
// masked with its bitmap word. `bsrc` is the bitmap (or, with no protected
// columns, any readable array of at least 4 words per block, and kmask = 0).
template <int S>
__device__ __forceinline__ float lane_tile(const LaneBlk<8, S> &t, cx16_ptr xb, cx4_ptr bsrc, uint32_t kmask,
                                           int64_t b, const uint4 *s_tab, float acc)
{
    const u32x4 bw = bsrc[b];
#pragma unroll
    for (int z = 0; z < 4; ++z) {
        const u32x16 xz = mask_group(xb[z], bw[z] & kmask);
        acc = lane_group<S>(t, z, xz, s_tab, acc);
        // finish each group before the next one (the compiler would otherwise
        // defer the products past the masking branches and keep every group's
        // table entries live)
        asm volatile("" : "+v"(acc));
    }
    return acc;
}

// The ragged last block of a row (d_in not a multiple of 128): activations
// past d_in read as zero.
template <int S>
__device__ __forceinline__ float lane_tile_ragged(const LaneBlk<8, S> &t, const uint32_t *x32, int64_t d_in,
                                                  cx4_ptr bsrc, uint32_t kmask, int64_t b, const uint4 *s_tab,
                                                  float acc)
{
    typedef const uint32_t __attribute__((address_space(4))) *cu32_ptr;
    const cu32_ptr xw = (cu32_ptr)(x32);
    const u32x4 bw = bsrc[b];
#pragma unroll
    for (int z = 0; z < 4; ++z) {
        u32x16 xz;
#pragma unroll
        for (int w = 0; w < 16; ++w) {
            const int64_t col = b * 128 + 32 * z + 2 * w;
            xz[w] = (col < d_in) ? xw[b * 64 + 16 * z + w] : 0u;
        }
        xz = mask_group(xz, bw[z] & kmask);
        acc = lane_group<S>(t, z, xz, s_tab, acc);
    }
    return acc;
}

// LoRA workgroup of the row-lane kernel: t_r = sum_j A[r][j] x_j (unmasked x)
// for one (member, rank index r), published into slot r of every row group
// of the member as a flagged 64-bit word for the group's finishing workgroup,
// which reads and clears it.
__device__ __forceinline__ void lane_lora_block(const GemvArgs &a, float *s_red)
{
    const int t = threadIdx.x;
    int m = 0;
    while (m + 1 < a.n && int64_t(blockIdx.x) >= a.mat[m + 1].lora_begin) ++m;
    const GemvMat &M = a.mat[m];
    const int r = int(int64_t(blockIdx.x) - M.lora_begin);
    // eight inputs per 16-byte load (x is 16-byte aligned; the row of A is
    // read in 16-byte pieces where it is, element by element where not),
    // four pieces per thread in flight
    const uint16_t *ar = M.A + int64_t(r) * a.d_in;
    const uint16_t *xr = static_cast<const uint16_t *>(a.x);
    const bool vec = ((reinterpret_cast<uintptr_t>(ar) & 15) == 0);
    const int64_t n8 = vec ? a.d_in / 8 : 0;
    float acc = 0.0f;
    for (int64_t p0 = t; p0 < n8; p0 += 4 * 256) {
        uint4 av[4], xv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t p = (p0 + u * 256 < n8) ? p0 + u * 256 : n8 - 1;
            av[u] = reinterpret_cast<const uint4 *>(ar)[p];
            xv[u] = reinterpret_cast<const uint4 *>(xr)[p];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            if (p0 + u * 256 >= n8) break;
            const uint32_t aw[4] = {av[u].x, av[u].y, av[u].z, av[u].w};
            const uint32_t xw[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                acc = __builtin_fmaf(__uint_as_float(aw[h] << 16), __uint_as_float(xw[h] << 16), acc);
                acc = __builtin_fmaf(__uint_as_float(aw[h] & 0xffff0000u), __uint_as_float(xw[h] & 0xffff0000u), acc);
            }
        }
    }
    for (int64_t j = n8 * 8 + t; j < a.d_in; j += 256)  // the rest, element by element
        acc = __builtin_fmaf(bf16_to_f32(ar[j]), bf16_to_f32(xr[j]), acc);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if ((t & 63) == 0) s_red[t >> 6] = acc;
    __syncthreads();
    const float tr = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
    const int64_t nrg = (M.d_out + 63) / 64;
    for (int64_t rg = t; rg < nrg; rg += 256)
        __hip_atomic_store(a.tslots + (M.rg_begin + rg) * BSQ_MAX_LORA_RANK + r,
                           (uint64_t(1) << 32) | __float_as_uint(tr), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The finishing workgroup's LoRA vector of row group rg: the LoRA
// workgroups' flagged slots (all loads in flight together, indices clamped
// to the rank), then cleared. Zeros when the member has no adapter.
__device__ __forceinline__ bool lane_lora_vector(const GemvArgs &a, const GemvMat &M, int64_t rg,
                                                 float (&tv)[BSQ_MAX_LORA_RANK])
{
#pragma unroll
    for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) tv[q] = 0.0f;
    if (M.rank == 0) return true;
    uint64_t *ts = a.tslots + (M.rg_begin + rg) * BSQ_MAX_LORA_RANK;
    uint64_t pw[BSQ_MAX_LORA_RANK];
    bool ok = true;
    for (int spin = 0;; ++spin) {
        if (spin >= a.spin_limit) {  // never expected: report, rather than hang
            ok = false;
            break;
        }
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q)
            pw[q] = __hip_atomic_load(ts + ((q < M.rank) ? q : M.rank - 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bool ready = true;
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) ready &= (pw[q] >> 32) != 0;
        if (__all(ready)) break;
        __builtin_amdgcn_s_sleep(1);
    }
#pragma unroll
    for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) tv[q] = (q < M.rank) ? __uint_as_float(uint32_t(pw[q])) : 0.0f;
    // the slots are cleared only when every one was consumed: after a give-up
    // a late flag may still land, so they stay as they are (the caller sees
    // the timeout bit and the poisoned workspace)
    const int lane = threadIdx.x & 63;
    if (ok && lane < M.rank) __hip_atomic_store(ts + lane, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return ok;
}

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

// c + <relu(lo + hi), u> over one pair of fp16 lanes (packed add and max,
// then v_dot2_f32_f16 with fp32 accumulation)
__device__ __forceinline__ float relu_dot2_f16(uint32_t lo, uint32_t hi, uint32_t u, float c)
{
    const half2_t pre = __builtin_bit_cast(half2_t, lo) + __builtin_bit_cast(half2_t, hi);
    const half2_t act = __builtin_elementwise_max(pre, half2_t{0, 0});
    return __builtin_amdgcn_fdot2(act, __builtin_bit_cast(half2_t, u), c, false);
}

// One tile of the d = 16 symmetric decoder (16 chunks of the lane's row, all
// stages). Per chunk and stage: the code's hidden pre-activation is the sum
// of the two split-table entries of its bytes (fp16, from LDS), the ReLU is
// taken in fp16, and the dot with the chunk's folded activation record (u in
// fp16, beta and the scale 2^e; staged in LDS for the workgroup's columns)
// is accumulated in fp32. `bl` is the tile's column block within the slice,
// `rch` the slice's chunks per stage.
template <int S>
__device__ __forceinline__ float lane_tile16(const LaneBlk<16, S> &t, const uint4 *s_rec, int rch, int bl,
                                             const uint4 *s_split, float acc)
{
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint4 cq = t.c[s][kk >> 3];
            const uint32_t cwd = ((kk & 7) >> 1) == 0 ? cq.x : ((kk & 7) >> 1) == 1 ? cq.y : ((kk & 7) >> 1) == 2 ? cq.z : cq.w;
            const uint32_t code = (kk & 1) ? (cwd >> 16) : (cwd & 0xffffu);
            // the chunk's record (LDS, wave-uniform address): u, then beta, 2^e
            const uint4 *rp = s_rec + (s * rch + bl * 16 + kk) * 4;
            const uint4 r0 = rp[0], r1 = rp[1];
            const uint2 r2 = *reinterpret_cast<const uint2 *>(rp + 2);
            // split tables [S][half][2][256] x 16 B: hidden units 0-7 and
            // 8-15 of a byte's entry are 4 KiB apart
            const uint4 *pl = s_split + (s * 4 + 0) * 256 + (code & 0xffu);
            const uint4 *ph = s_split + (s * 4 + 2) * 256 + (code >> 8);
            const uint4 l0 = pl[0], l1 = pl[256], h0 = ph[0], h1 = ph[256];
            const uint32_t lw[8] = {l0.x, l0.y, l0.z, l0.w, l1.x, l1.y, l1.z, l1.w};
            const uint32_t hw[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
            // (the words are bit-cast inside a helper: bit-casting elements of a
            // scalar-loaded vector in place was once compiled to read element 0
            // for every pair)
            const uint32_t rw[10] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w, r2.x, r2.y};
            float dsum = __uint_as_float(rw[8]);
#pragma unroll
            for (int i = 0; i < 8; ++i) dsum = relu_dot2_f16(lw[i], hw[i], rw[i], dsum);
            dsum *= __uint_as_float(rw[9]);
            const uint4 gq = t.g[s][kk >> 3];
            const uint32_t gw = ((kk & 7) >> 1) == 0 ? gq.x : ((kk & 7) >> 1) == 1 ? gq.y : ((kk & 7) >> 1) == 2 ? gq.z : gq.w;
            const float gv = (kk & 1) ? half_hi(gw) : half_lo(gw);
            acc = __builtin_fmaf(gv, dsum, acc);
        }
        asm volatile("" : "+v"(acc));  // one chunk's entries and record live at a time
    }
    return acc;
}

template <int D, int S, int TPW>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(S <= 2 ? 4 : 2))) void gemv_lane_kernel(
    const GemvArgs a)
{
    constexpr int WV = 4, NT = 256;      // waves per workgroup, threads
    constexpr int PF = TPW < 2 ? TPW : 2;  // tiles in flight per wave
    // LDS table: d = 8, [S][256] bf16 decoder entries (16 B); d = 16, the
    // split pre-activation tables [S][2][2][256] (16 B groups)
    constexpr int TAB = (D == 8) ? S * 256 : S * 1024;  // uint4 units
    // d = 16: the folded activation records of the slice's columns,
    // [S][RCH chunks] 64-byte slots
    constexpr int RCH = WV * TPW * 16;
    constexpr int REC = (D == 8) ? 0 : S * RCH * 4;  // uint4 units
    // the table in static LDS (its address is a constant the compiler folds
    // into each lookup's offset), the rest in the dynamic allocation
    __shared__ __attribute__((aligned(16))) uint4 s_tab_mem[TAB];
    extern __shared__ uint4 s_mem[];
    uint4 *s_tab = s_tab_mem;
    uint4 *s_rec = s_mem;
    float *s_red = reinterpret_cast<float *>(s_mem + REC);  // [WV][64] wave sums
    float *s_xs = s_red + WV * 64;                             // [kp] scale_p * x_{idx_p}
    const int64_t kp = q8_pitch(a.k);
    int8_t *s_q8 = reinterpret_cast<int8_t *>(s_xs + kp);      // [64][kp] int8 rows (finishing slice)
    const bool q8_lds = kp <= LANE_Q8_LDS_MAX;
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);

    // The kernel arguments reach the workgroup by scalar loads whose round
    // trips would add up if each waited for the one before: the member comes
    // from the first blocks of all members (one batch of loads), then the
    // member's pointers that the prologue needs are read together (a second
    // batch), each batch forced to complete at once by an empty asm that
    // takes the values.
    const int32_t bid = int32_t(blockIdx.x) - a.lora_blocks32;
    int m = 0;
    int32_t bbm = 0;  // the member's first block (a.bb[m], selected, not reloaded)
#pragma unroll
    for (int i = 1; i < BSQ_MAX_GROUP; ++i) {
        const int32_t bbi = a.bb[i];
        m += (bid >= bbi) ? 1 : 0;
        bbm = (bid >= bbi) ? bbi : bbm;
    }
    {
        const int64_t nb_ = a.nblk, q_ = a.q, k_ = a.k, din_ = a.d_in;
        const void *x_ = a.x;
        asm volatile("" ::"s"(m), "s"(nb_), "s"(q_), "s"(k_), "s"(din_), "s"(x_));
    }
    if (bid < 0) {  // the LoRA vectors, ahead of every tile
        lane_lora_block(a, reinterpret_cast<float *>(s_mem));
        return;
    }
    const GemvMat &M = a.mat[m];
    LanePlanes<S> PL;
#pragma unroll
    for (int s = 0; s < S; ++s) {
        PL.codes[s] = static_cast<const uint8_t *>(M.codes[s]);
        PL.gains[s] = M.gains[s];
    }
    const uint4 *tabp[S];
#pragma unroll
    for (int s = 0; s < S; ++s)
        tabp[s] = (D == 8) ? reinterpret_cast<const uint4 *>(M.tab16[s]) : reinterpret_cast<const uint4 *>(M.split[s]);
    const int8_t *q8p = M.q8;
    const int32_t *idxp = M.idx;
    const float *scalep = M.scale;
    const int64_t d_out_m = M.d_out;
    asm volatile("" ::"s"(PL.codes[0]), "s"(PL.gains[0]), "s"(tabp[0]), "s"(q8p), "s"(idxp), "s"(scalep),
                 "s"(d_out_m));
    if constexpr (S > 1) asm volatile("" ::"s"(PL.codes[S - 1]), "s"(PL.gains[S - 1]), "s"(tabp[S - 1]));
    // Prologue in a fixed issue order (vector-memory completions are counted
    // in order): the decoder table straight to LDS by DMA
    // (global_load_lds_dwordx4, 64 entries per wave instruction), then the
    // first tiles, so that the wait before the barrier covers the table but
    // not the tiles. Tile indices are clamped so every load is in bounds and
    // unconditional (a wave without tiles reloads its row group's first tile).
    // The table goes first, before the workgroup's index arithmetic.
    static_assert(TAB % NT == 0, "table chunks are shared out evenly");
#pragma unroll
    for (int r = 0; r < TAB / NT; ++r) {
        const int c = r * WV + wave;  // 1 KiB chunk of the table: 64 lanes x 16 B
        const uint4 *src = (D == 8) ? tabp[c >> 2] + (c & 3) * 64 + lane : tabp[c >> 4] + (c & 15) * 64 + lane;
        __builtin_amdgcn_global_load_lds(src, s_tab + c * 64, 16, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    const int64_t nblk = a.nblk, Q = a.q;
    const int32_t unit = bid - bbm;  // row group * Q + slice
    const int64_t rg = uint32_t(unit) / uint32_t(Q), q = unit - rg * Q;
    const int64_t tbase = ((rg * nblk) << 10) + (int64_t(lane) << 4);
    // this wave's tiles [b0, b1); those whose 128 columns are all real go
    // through the pipelined loop, a ragged last tile of the row (d_in not a
    // multiple of 128) is handled after it
    const int64_t full_blocks = (D == 8) ? (a.d_in / 8) / 16 : nblk;  // d = 16: padding chunks read zeros
    // the row group's nblk tiles are shared out evenly over its Q * WV waves
    // (floor or ceil of nblk / (Q WV) each, at most TPW), in order, so no wave
    // is left idle while another carries a whole extra tile set
    const int64_t nw = Q * WV, wq = q * WV + wave;
    const int64_t b0 = uint32_t(wq * nblk) / uint32_t(nw);  // (products below 2^31: checked at launch)
    const int64_t b1 = uint32_t((wq + 1) * nblk) / uint32_t(nw);
    const int64_t sb0 = uint32_t(q * nblk) / uint32_t(Q);  // the slice's first block (wave 0's b0)
    const int64_t nt = ((b1 < full_blocks) ? b1 : full_blocks) - b0;  // may be <= 0
    const bool ragged = b0 <= full_blocks && full_blocks < b1;
    const bool fin = q == Q - 1;  // this slice finishes the row group

    if constexpr (D == 16) {
        // the slice's records, 16 per wave instruction (four lanes per 64-byte
        // slot); chunks past the row's padded end read the last slot (unused)
        static_assert((S * RCH / 16) % WV == 0, "record chunks are shared out evenly");
        const int64_t c0 = sb0 * 16;  // the slice's first chunk (the slice spans at most RCH chunks)
#pragma unroll
        for (int r = 0; r < S * RCH / 16 / WV; ++r) {
            const int e = r * WV + wave;
            const int s = e / (RCH / 16);
            const int64_t cc = c0 + (e % (RCH / 16)) * 16 + lane / 4;
            const uint4 *src = reinterpret_cast<const uint4 *>(
                M.xp + (int64_t(s) * a.pitch + ((cc < a.pitch) ? cc : a.pitch - 1)) * 16) + (lane & 3);
            __builtin_amdgcn_global_load_lds(src, s_rec + e * 64, 16, 0, 0);
        }
    }
    // the finishing slice brings its row group's int8 rows to LDS the same way
    // (rows past d_out get clamped copies and are never read)
    if (fin && a.k > 0 && q8_lds) {
        const int8_t *src = q8p + rg * 64 * kp;
        const int64_t avail = ((d_out_m - rg * 64 < 64) ? d_out_m - rg * 64 : 64) * kp;
        for (int64_t o = int64_t(wave) * 1024; o < 64 * kp; o += WV * 1024) {
            const int64_t e = o + lane * 16;
            const int64_t es = (e < avail) ? e : avail - 16;
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const uint4 *>(src + es), s_q8 + o, 16, 0, 0);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // a wave without a full tile works on the slice's first block (always a
    // real block) and drops the result
    const int64_t blast = (nt > 0) ? b0 + nt - 1 : sb0;
    LaneBlk<D, S> buf[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u) lane_load<D, S>(buf[u], PL, tbase + (((b0 + u < blast) ? b0 + u : blast) << 10));
    __builtin_amdgcn_sched_barrier(0);
    // protected index and scale of this thread's column, used at the end
    // (unconditional loads, so that every path has the same loads in flight;
    // with no protected columns they read x and are ignored)
    const int64_t pt = (a.k > 0) ? ((t < a.k) ? t : a.k - 1) : 0;
    const int32_t pj_raw = ((a.k > 0) ? idxp : static_cast<const int32_t *>(a.x))[pt];
    const float psc = ((a.k > 0) ? scalep : static_cast<const float *>(a.x))[pt];
    const int32_t pj = (a.k > 0) ? pj_raw : -1;
    // the workspace's poison word, read by the finishing slice before it
    // consumes any slot (unconditional, like the loads above)
    const uint32_t poisoned = __hip_atomic_load(a.poison, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the table is in LDS once at most the tile, index and poison loads are
    // pending; a plain s_barrier (no release fence) lets those stay in flight
    constexpr int NIDX = PF * (D / 8 + 2) * S + 3;
    __builtin_amdgcn_s_waitcnt((NIDX & 15) | ((NIDX >> 4) << 14) | (7 << 4) | (15 << 8));
    asm volatile("s_barrier" ::: "memory");

    const cx16_ptr xv = (cx16_ptr)(a.x);
    // the bitmap, or (no protected columns) x itself read under a zero mask,
    // so that the per-tile bitmap load is unconditional
    const cx4_ptr bsrc = (a.k > 0) ? (cx4_ptr)(M.bits) : (cx4_ptr)(a.x);
    const uint32_t kmask = (a.k > 0) ? ~0u : 0u;
    // the wave's tiles as straight-line code with PF tiles in flight (no
    // loop, so the waits before each tile count exactly the loads issued
    // after it); tile indices are clamped to the wave's last full tile so
    // every load is unconditional, and the tiles past nt (a wave with one
    // tile fewer than TPW, or none) are loaded but not computed
    float acc = 0.0f;
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        const int64_t b = (b0 + u < blast) ? b0 + u : blast;
        if (u < nt) {
            if constexpr (D == 8) acc += lane_tile<S>(buf[u % PF], xv + 4 * b, bsrc, kmask, b, s_tab, 0.0f);
            else acc += lane_tile16<S>(buf[u % PF], s_rec, RCH, int(b - sb0), s_tab, 0.0f);
        }
        if (u + PF < TPW)
            lane_load<D, S>(buf[u % PF], PL, tbase + (((b0 + u + PF < blast) ? b0 + u + PF : blast) << 10));
    }
    if constexpr (D == 8) {
        if (ragged) {
            const int64_t b = full_blocks;
            lane_load<D, S>(buf[0], PL, tbase + (b << 10));
            acc = lane_tile_ragged<S>(buf[0], static_cast<const uint32_t *>(a.x), a.d_in, bsrc, kmask, b, s_tab,
                                      acc);
        }
    }

    // the finishing slice's protected columns: the scaled activations to LDS
    // (indices loaded above), then each wave adds every fourth 16-column
    // word of its lane's row to its own sum (the four shares are added with
    // the wave sums, in wave order), off the finishing wave's serial path
    if (fin && a.k > 0) {
        if (t < kp) s_xs[t] = (t < a.k && pj >= 0 && pj < a.d_in) ? psc * load_x(a.x, pj, 1) : 0.0f;
        for (int64_t p = NT + t; p < kp; p += NT) {  // more protected columns than threads
            const int32_t j = (p < a.k) ? M.idx[p] : -1;
            s_xs[p] = (j >= 0 && j < a.d_in) ? M.scale[p] * load_x(a.x, j, 1) : 0.0f;
        }
        __syncthreads();
        const int64_t row_w = rg * 64 + lane;
        if (row_w < M.d_out) acc = lane_q8_term(a, M, s_xs, s_q8, q8_lds, row_w, wave, WV, acc);
    }
    // the four wave sums of each row, in wave order
    s_red[wave * 64 + lane] = acc;
    __syncthreads();
    if (wave != 0) return;
    float v = s_red[lane];
#pragma unroll
    for (int w = 1; w < WV; ++w) v += s_red[w * 64 + lane];
    const int64_t row = rg * 64 + lane;
    uint64_t *slots = a.slots + (M.rg_begin + rg) * (Q - 1) * 64 + lane;
    if (!fin) {
        __hip_atomic_store(slots + q * 64, (uint64_t(1) << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        return;
    }
    // a workspace poisoned by an earlier call that gave up waiting may hold
    // flags that no slice of this call wrote: consume nothing, write NaN and
    // report (the caller zero-fills the workspace to recover)
    if (poisoned != 0u) {
        if (lane == 0 && a.err) atomicOr(a.err, int32_t(BSQ_DEVERR_POISONED));
        if (row < M.d_out) lane_store(a, M, row, __builtin_nanf(""));
        return;
    }
    // the finishing slice adds the LoRA term to its own sum (and protected
    // shares) first: it does not depend on the other slices, so this work
    // overlaps the wait for them
    float tv[BSQ_MAX_LORA_RANK];
    const bool ok = lane_lora_vector(a, M, rg, tv);
    if (row < M.d_out) v = lane_lora_term(M, row, v, tv);
    float tot = 0.0f;
    bool timed_out = false;
    // the other slices' slots, eight at a time, all eight loads in flight
    // together (slot indices clamped to the last one, extra copies unused)
    constexpr int PW = 8;
    for (int64_t q0 = 0; q0 < Q - 1 && !timed_out; q0 += PW) {
        uint64_t pw[PW];
        for (int spin = 0;; ++spin) {
            if (spin >= a.spin_limit) {  // never expected: report, rather than hang
                timed_out = true;
                break;
            }
#pragma unroll
            for (int u = 0; u < PW; ++u)
                pw[u] = __hip_atomic_load(slots + ((q0 + u < Q - 1) ? q0 + u : Q - 2) * 64, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
            bool ready = true;
#pragma unroll
            for (int u = 0; u < PW; ++u) ready &= (pw[u] >> 32) != 0;
            if (__all(ready)) break;
            __builtin_amdgcn_s_sleep(1);
        }
#pragma unroll
        for (int u = 0; u < PW; ++u) tot += (q0 + u < Q - 1) ? __uint_as_float(uint32_t(pw[u])) : 0.0f;
    }
    tot += v;
    if (timed_out || !ok) {
        // a slice that is late may still set its flag: leave every slot as it
        // is and mark the workspace, so that no later call takes such a flag
        // for one of its own
        if (lane == 0) {
            __hip_atomic_store(a.poison, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a.err) atomicOr(a.err, int32_t(BSQ_DEVERR_TIMEOUT));
        }
        if (row < M.d_out) lane_store(a, M, row, __builtin_nanf(""));
        return;
    }
    for (int64_t q0 = 0; q0 < Q - 1; ++q0)
        __hip_atomic_store(slots + q0 * 64, uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (row < M.d_out) lane_store(a, M, row, tot);
}

// ---------------------------------------------------------------------------
// fp32 activations: the fp32 decoder table and fp32 arithmetic throughout.
// One wave per row, lanes stride over the chunks.
// ---------------------------------------------------------------------------
// fp32 arithmetic throughout (fp32 x, and every configuration with b != d,
// whatever the dtype of x): one wave per row over the 2^B-entry fp32 table,
// D inputs per chunk and B code bits per stage; lanes stride the chunks.
template <int D, int B, int S>
__global__ __launch_bounds__(256) void gemv_f32_kernel(const GemvArgs a)
{
    const int lane = threadIdx.x & 63;
    const int64_t wave = (int64_t(blockIdx.x) * blockDim.x + threadIdx.x) >> 6;
    int m = 0;
    int64_t row = wave;
    while (m < a.n && row >= a.mat[m].d_out) {
        row -= a.mat[m].d_out;
        ++m;
    }
    if (m >= a.n) return;
    const GemvMat &M = a.mat[m];
    const int64_t C = a.d_in / D;
    float acc = 0.0f;
    for (int64_t c = lane; c < C; c += 64) {
        float xv[D];
        // protected inputs of the chunk: from the bitmap when the layer has
        // one (one word per chunk, D divides 32), else by search of the list
        uint32_t pm = 0;
        if (a.k > 0 && M.bits) pm = (M.bits[(c * D) >> 5] >> ((c * D) & 31)) & uint32_t((uint64_t(1) << D) - 1u);
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int64_t col = c * D + j;
            const bool prot = M.bits ? ((pm >> j) & 1u) : (a.k > 0 && is_protected(M.idx, a.k, col));
            xv[j] = prot ? 0.0f : load_x(a.x, col, a.x_bf16);
        }
        const int64_t off = tile_index(row, c, a.pitch);
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint32_t code = (B == 8) ? uint32_t(static_cast<const uint8_t *>(M.codes[s])[off])
                                           : uint32_t(static_cast<const uint16_t *>(M.codes[s])[off]);
            const float gs = f16_bits_to_f32(M.gains[s][off]);
            const float *y = M.tab32[s] + size_t(code) * D;
            float dsum = 0.0f;
#pragma unroll
            for (int j = 0; j < D; ++j) dsum = __builtin_fmaf(y[j], xv[j], dsum);
            acc = __builtin_fmaf(gs, dsum, acc);
        }
    }
    for (int64_t p = lane; p < a.k; p += 64)
        acc = __builtin_fmaf(payload_to_f32(uint8_t(M.q8[row * q8_pitch(a.k) + p]), a.pfmt),
                             M.scale[p] * load_x(a.x, M.idx[p], a.x_bf16), acc);
    for (int q = lane; q < M.rank; q += 64) acc = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], acc);
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) {
        if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(acc);
        else static_cast<float *>(M.y)[row] = acc;
    }
}

template <int D, int B>
hipError_t launch_f32(int stages, const GemvArgs &a, int64_t rows, hipStream_t st)
{
    const dim3 grid(unsigned((rows + 3) / 4));
    switch (stages) {
    case 1: hipLaunchKernelGGL((gemv_f32_kernel<D, B, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemv_f32_kernel<D, B, 2>), grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemv_f32_kernel<D, B, 3>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((gemv_f32_kernel<D, B, 4>), grid, dim3(256), 0, st, a); break;
    }
    return hipGetLastError();
}

template <int D>
hipError_t launch_stream(int stages, const GemvArgs &a, int nt, int grid, size_t shm, hipStream_t st)
{
    switch (stages) {
    case 1: hipLaunchKernelGGL((gemv_stream_kernel<D, 1>), dim3(grid), dim3(nt), shm, st, a); break;
    case 2: hipLaunchKernelGGL((gemv_stream_kernel<D, 2>), dim3(grid), dim3(nt), shm, st, a); break;
    case 3: hipLaunchKernelGGL((gemv_stream_kernel<D, 3>), dim3(grid), dim3(nt), shm, st, a); break;
    default: hipLaunchKernelGGL((gemv_stream_kernel<D, 4>), dim3(grid), dim3(nt), shm, st, a); break;
    }
    return hipGetLastError();
}

template <int D, int TPW>
void launch_lane(int stages, const GemvArgs &a, int64_t blocks, size_t shm, hipStream_t st)
{
    const dim3 grid{unsigned(blocks)}, blk{256u};
    switch (stages) {
    case 1: hipLaunchKernelGGL((gemv_lane_kernel<D, 1, TPW>), grid, blk, shm, st, a); break;
    case 2: hipLaunchKernelGGL((gemv_lane_kernel<D, 2, TPW>), grid, blk, shm, st, a); break;
    case 3: hipLaunchKernelGGL((gemv_lane_kernel<D, 3, TPW>), grid, blk, shm, st, a); break;
    default: hipLaunchKernelGGL((gemv_lane_kernel<D, 4, TPW>), grid, blk, shm, st, a); break;
    }
}

GemvArgs make_args(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                   const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype, void *ws,
                   bool scratch_layout)
{
    GemvArgs a{};
    a.n = n;
    a.d_in = layers[0].d_in;
    a.pitch = layers[0].pitch;
    a.k = layers[0].k;
    a.x = x;
    a.x_bf16 = (x_dtype == BSQ_BF16);
    a.y_bf16 = (y_dtype == BSQ_BF16);
    a.stages = cfg.stages;
    char *wb = static_cast<char *>(ws) + GEMV_HDR;
    float *wt = reinterpret_cast<float *>(wb);
    a.poison = static_cast<uint32_t *>(ws);
    a.spin_limit = wait_limit();
    a.pfmt = cfg.protect_format;
    // workspace of one configuration: header, LoRA vectors, folded activation
    // records, slots. The shared scratch array of bsq_gemv_noalloc keeps the
    // records in its last GEMV_SCRATCH_XP_BYTES instead, so that the slots of
    // every configuration start at the same offset and never overlap records
    char *xp_base = scratch_layout ? static_cast<char *>(ws) + (BSQ_GEMV_NOALLOC_SCRATCH_BYTES - GEMV_SCRATCH_XP_BYTES)
                                   : wb + gemv_t_bytes();
    a.slots = reinterpret_cast<uint64_t *>(wb + gemv_t_bytes() + (scratch_layout ? 0 : gemv_xp_bytes(cfg, a.pitch)));
    for (int m = 0; m < n; ++m) {
        GemvMat &M = a.mat[m];
        const bsq_layer &L = layers[m];
        const char *cb = codecs ? static_cast<const char *>(codecs[m]) : nullptr;
        for (int s = 0; s < cfg.stages; ++s) {
            M.codes[s] = L.codes[s];
            M.gains[s] = L.gains[s];
            if (cb) {
                M.tab16[s] = reinterpret_cast<const uint16_t *>(cb + codec_tab16_offset(cfg, s));
                M.tab32[s] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, s));
                if (codec_has_split(cfg)) {
                    M.split[s] = reinterpret_cast<const uint16_t *>(cb + codec_split_offset(cfg, s));
                    M.w2[s] = reinterpret_cast<const float *>(cb + codec_w2_offset(cfg, s));
                    M.b2[s] = reinterpret_cast<const float *>(cb + codec_b2_offset(cfg, s));
                }
            }
        }
        M.xp = reinterpret_cast<uint32_t *>(xp_base) + int64_t(m) * cfg.stages * a.pitch * 16;
        M.idx = L.prot_idx;
        M.q8 = L.prot_q8;
        M.scale = L.prot_scale;
        M.bits = L.prot_bits;
        M.rank = 0;
        if (loras && loras[m].rank > 0) {
            M.A = loras[m].A;
            M.B = loras[m].B;
            M.rank = loras[m].rank;
        }
        M.d_out = L.d_out;
        M.y = y ? y[m] : nullptr;
        M.t = wt + m * BSQ_MAX_LORA_RANK;
    }
    return a;
}

}  // namespace

// Row-lane kernel: a workgroup (4 waves) covers up to 4 * TPW consecutive
// tiles of one 64-row group, so a row group has Q = ceil(nblk / (4 TPW))
// slices, its nblk tiles shared evenly over the Q * 4 waves.
// LANE_MIN_WAVES is half of the 4096 wave slots of 256 compute units at
// four waves per SIMD.
constexpr int64_t LANE_MIN_WAVES = 2048;

int64_t lane_slices(int64_t nblk, int tpw) { return (nblk + 4 * tpw - 1) / (4 * tpw); }

int lane_tpw(int64_t row_groups, int64_t nblk)
{
    // two tiles per wave measured fastest on the Qwen3-shaped launches
    // (1024 to 51200 rows, 4096 to 25600 inputs), with the tiles shared out
    // evenly; one where two would leave fewer than LANE_MIN_WAVES waves
    return (row_groups * lane_slices(nblk, 2) * 4 >= LANE_MIN_WAVES) ? 2 : 1;
}

size_t gemv_ws_bytes(const bsq_config &cfg, int64_t n, int64_t max_d_out, int64_t d_in)
{
    const int64_t rg = n * ((max_d_out + 63) / 64);
    const int64_t nblk = (d_in / cfg.d + BSQ_PITCH_ALIGN - 1) / BSQ_PITCH_ALIGN;
    // LoRA vectors, folded activation records (d = 16 decoder path), then
    // {flag, partial} slots for all but the last slice (as many slices as the
    // smallest TPW makes), then the flagged LoRA vector slots of every row
    // group
    return GEMV_HDR + gemv_t_bytes() + gemv_xp_bytes(cfg, nblk * BSQ_PITCH_ALIGN) +
           size_t(rg) * size_t(lane_slices(nblk, 1) - 1) * 64 * 8 + size_t(rg) * BSQ_MAX_LORA_RANK * 8;
}

bool gemv_scratch_fits(const bsq_config &cfg, int64_t n, int64_t max_d_out, int64_t d_in)
{
    const int64_t nblk = (d_in / cfg.d + BSQ_PITCH_ALIGN - 1) / BSQ_PITCH_ALIGN;
    const size_t xp = gemv_xp_bytes(cfg, nblk * BSQ_PITCH_ALIGN);
    return xp <= GEMV_SCRATCH_XP_BYTES &&
           gemv_ws_bytes(cfg, n, max_d_out, d_in) - xp <= BSQ_GEMV_NOALLOC_SCRATCH_BYTES - GEMV_SCRATCH_XP_BYTES;
}

size_t gemv_stream_lds_bytes(const bsq_config &cfg, int64_t d_in, int64_t nseg_rpb)
{
    const int64_t words = (d_in + 31) / 32;
    const int64_t k = cfg.protect_num ? (d_in * cfg.protect_num + cfg.protect_den - 1) / cfg.protect_den : 0;
    return ((cfg.d == 8) ? size_t(cfg.stages) * 256 * 16 : 0) + size_t(nseg_rpb) * 4 +
           size_t((words + 3) & ~int64_t(3)) * 4 + size_t(k) * 4;
}

hipError_t launch_gemv_prep(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                            const bsq_lora *loras, const void *x, int x_dtype, void *ws, bool scratch_layout,
                            hipStream_t st)
{
    bool any = false;
    for (int m = 0; m < n && loras; ++m) any |= (loras[m].rank > 0);
    // the row-lane kernel computes its LoRA vectors itself
    if (gemv_lane_path(cfg, x_dtype)) any = false;
    const bool fold = gemv_split16(cfg) && x_dtype == BSQ_BF16;
    if (!any && !fold) return hipSuccess;
    const GemvArgs a = make_args(cfg, n, codecs, layers, loras, x, x_dtype, nullptr, BSQ_F32, ws, scratch_layout);
    const int lora_blocks = any ? n * BSQ_MAX_LORA_RANK : 0;
    const int64_t fold_blocks = fold ? int64_t(n) * cfg.stages * (a.pitch / 16) : 0;
    hipLaunchKernelGGL(gemv_prep_kernel, dim3(unsigned(lora_blocks + fold_blocks)), dim3(256), 0, st, a, lora_blocks);
    return hipGetLastError();
}

hipError_t launch_gemv_run(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                           const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype,
                           void *ws, bool scratch_layout, int32_t *err, hipStream_t st)
{
    const int D = cfg.d, S = cfg.stages;
    GemvArgs a = make_args(cfg, n, codecs, layers, loras, x, x_dtype, y, y_dtype, ws, scratch_layout);
    a.err = err;
    int64_t rows_total = 0;
    for (int m = 0; m < n; ++m) rows_total += layers[m].d_out;
    if (rows_total == 0) return hipSuccess;
    if (x_dtype != BSQ_BF16 || cfg.b != cfg.d) {
        if (cfg.b == cfg.d)
            return (D == 8) ? launch_f32<8, 8>(S, a, rows_total, st) : launch_f32<16, 16>(S, a, rows_total, st);
        return (D == 8) ? launch_f32<8, 16>(S, a, rows_total, st) : launch_f32<16, 8>(S, a, rows_total, st);
    }

    if (D == 8 || gemv_split16(cfg)) {
        // row-lane kernel: one workgroup per (64-row group, slice of tiles)
        a.nblk = a.pitch / 16;
        int64_t rgs = 0;
        for (int m = 0; m < n; ++m) rgs += (layers[m].d_out + 63) / 64;
        const int tpw = lane_tpw(rgs, a.nblk);
        a.q = lane_slices(a.nblk, tpw);
        // LoRA workgroups first (one per member and rank index), then the
        // tiles' workgroups; the LoRA vector slots follow the partial slots
        a.tslots = a.slots + rgs * (lane_slices(a.nblk, 1) - 1) * 64;
        int64_t blocks = 0, lora_blocks = 0;
        rgs = 0;
        for (int m = 0; m < n; ++m) {
            const int64_t nrg = (layers[m].d_out + 63) / 64;
            a.mat[m].block_begin = blocks;
            a.mat[m].rg_begin = rgs;
            a.mat[m].lora_begin = lora_blocks;
            blocks += nrg * a.q;
            rgs += nrg;
            lora_blocks += a.mat[m].rank;
        }
        a.lora_blocks = lora_blocks;
        blocks += lora_blocks;
        if (blocks > INT32_MAX || a.q * 4 * a.nblk > INT32_MAX) return hipErrorInvalidConfiguration;
        a.lora_blocks32 = int32_t(lora_blocks);
        for (int m = 0; m < BSQ_MAX_GROUP; ++m) a.bb[m] = (m < n) ? int32_t(a.mat[m].block_begin) : INT32_MAX;
        const int64_t kp = q8_pitch(a.k);
        // dynamic LDS: the d = 16 records, wave sums, scaled protected
        // activations, the finishing slice's int8 rows (the table is static)
        const size_t rec = (D == 8) ? 0 : size_t(S) * 4 * tpw * 16 * 64;
        const size_t shm = rec + 4 * 64 * 4 + size_t(kp) * 4 + ((kp <= LANE_Q8_LDS_MAX) ? size_t(64 * kp) : 0);
        if (D == 8) {
            switch (tpw) {
            case 8: launch_lane<8, 8>(S, a, blocks, shm, st); break;
            case 6: launch_lane<8, 6>(S, a, blocks, shm, st); break;
            case 5: launch_lane<8, 5>(S, a, blocks, shm, st); break;
            case 4: launch_lane<8, 4>(S, a, blocks, shm, st); break;
            case 3: launch_lane<8, 3>(S, a, blocks, shm, st); break;
            case 2: launch_lane<8, 2>(S, a, blocks, shm, st); break;
            default: launch_lane<8, 1>(S, a, blocks, shm, st); break;
            }
        } else {
            switch (tpw) {
            case 4: launch_lane<16, 4>(S, a, blocks, shm, st); break;
            case 2: launch_lane<16, 2>(S, a, blocks, shm, st); break;
            default: launch_lane<16, 1>(S, a, blocks, shm, st); break;
            }
        }
        return hipGetLastError();
    }
    const int64_t nseg = a.pitch / (128 / D);
    // block size: the multiple of 64 up to 512 that leaves the fewest idle threads
    int nt = 256;
    double best = -1.0;
    for (int cand = 64; cand <= 512; cand += 64) {
        if (nseg > cand) continue;
        const double use = double((cand / nseg) * nseg) / cand;
        if (use > best + 1e-9 || (use > best - 1e-9 && cand == 256)) {
            best = use;
            nt = cand;
        }
    }
    const int64_t rs = nt / nseg;
    // rows per thread: enough rows per block that every thread reuses its x~
    // segment, while keeping about three blocks per compute unit busy
    const int64_t target_blocks = 768;
    int64_t rpt = (rows_total + rs * target_blocks - 1) / (rs * target_blocks);
    if (rpt < 1) rpt = 1;
    if (rpt > 16) rpt = 16;
    while (rpt > 1 && rs * rpt * nseg * 4 > 32768) --rpt;
    a.nseg = nseg;
    a.rs = rs;
    a.rpb = rs * rpt;
    int64_t blocks = 0;
    for (int m = 0; m < n; ++m) {
        a.mat[m].block_begin = blocks;
        blocks += (layers[m].d_out + a.rpb - 1) / a.rpb;
    }
    const size_t shm = gemv_stream_lds_bytes(cfg, a.d_in, a.rpb * nseg);
    return launch_stream<16>(S, a, nt, int(blocks), shm, st);
}

// ---------------------------------------------------------------------------
// The library-owned GEMV workspace of bsq_gemv_noalloc: one file-scope device
// array per GPU. In host code `scratch` only names the symbol; the kernels get
// its device address, taken once per device with hipGetSymbolAddress while
// that device is current.
// ---------------------------------------------------------------------------
namespace {

static __device__ __align__(256) uint8_t scratch[BSQ_GEMV_NOALLOC_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[SCRATCH_MAX_DEVICES];
bool g_scratch_cleared[SCRATCH_MAX_DEVICES];

// zero-fill of the scratch array (a kernel, not a memset, so that a call
// captured into a graph replays it correctly)
__global__ __launch_bounds__(256) void scratch_clear_kernel(uint4 *p, int64_t n16)
{
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n16; i += int64_t(gridDim.x) * 256)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

}  // namespace

hipError_t gemv_scratch(bool clear, void **ptr, hipStream_t st)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return hipErrorInvalidDevice;
    bool first = false;
    {
        std::lock_guard<std::mutex> lock(g_scratch_mutex);
        if (!g_scratch_ptr[dev]) {
            void *p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (!p || (reinterpret_cast<uintptr_t>(p) & 255)) return hipErrorInvalidSymbol;
            g_scratch_ptr[dev] = p;
        }
        first = !g_scratch_cleared[dev];
        g_scratch_cleared[dev] = true;
        *ptr = g_scratch_ptr[dev];
    }
    if (first || clear) {
        constexpr int64_t n16 = int64_t(BSQ_GEMV_NOALLOC_SCRATCH_BYTES) / 16;
        hipLaunchKernelGGL(scratch_clear_kernel, dim3(unsigned(n16 / 256 / 16)), dim3(256), 0, st,
                           static_cast<uint4 *>(*ptr), n16);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace bsq
