// Fused decode-GEMV at batch 1 (the direct computation from binary spherical
// codes that Section V names as future work):
//   y_i = sum_c sum_s gain_s(i,c) * <D_s(code_s(i,c)), x~_c>
//         + sum_p q8(i,p) * (scale_p x_{idx_p}) + sum_r B(i,r) (A x)_r
// where x~ is x with the protected input columns zeroed (those columns come
// from the int8 path, eq. protected_8bit_scatter) and the stage sum is the
// parallel residual decoding of eq. parallel_stage_decode.
//
// Streaming kernel (bf16 activations). Each block owns a contiguous range of
// rows of one group member. At start it stages in LDS the member's bf16
// decoder table (d = 8), the protected-column bitmap and the scaled protected
// activations scale_p * x_{idx_p}. A thread owns one 128-input segment of x~
// (16 chunks at d = 8, 8 chunks at d = 16), masked and held in registers,
// and walks down its rows two at a time: the next row's code and gain words
// (128-bit loads, read once from HBM) are in flight while the current row is
// decoded by table lookup and dotted with x~ by v_dot2_f32_bf16 in fp32.
// Segment partials go to LDS and are reduced once per block, where the
// epilogue adds the int8 and LoRA terms. The only other kernel is the LoRA
// prep (t = A x, one fp32 16-vector per member), launched only when a member
// has an adapter.
#include "bsq_internal.h"

namespace bsq {
namespace {

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
    int64_t d_out;
    int64_t block_begin;  // first block of this member in the streaming grid
    float *t;             // workspace: A x, [16]
    void *y;
};

struct GemvArgs {
    GemvMat mat[BSQ_MAX_GROUP];
    int n;
    int64_t d_in, pitch, k, nseg, rs, rpb;
    const void *x;
    int x_bf16, y_bf16;
};

__device__ __forceinline__ float load_x(const void *x, int64_t j, int bf)
{
    return bf ? bf16_to_f32(static_cast<const uint16_t *>(x)[j]) : static_cast<const float *>(x)[j];
}

// ---------------------------------------------------------------------------
// LoRA prep: t[m][r] = sum_j A[r][j] x_j (unmasked x), one block per (m, r).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemv_lora_prep_kernel(const GemvArgs a)
{
    __shared__ float red[256];
    const int m = blockIdx.x / BSQ_MAX_LORA_RANK;
    const int r = blockIdx.x % BSQ_MAX_LORA_RANK;
    const int t = threadIdx.x;
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

    // block setup: decoder table, protected bitmap, scaled protected activations
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

    const int slot = t / nseg, seg = t - slot * nseg;
    if (slot < rs) {
        // x~ segment: 128 bf16 inputs starting at seg * 128, protected positions zeroed
        uint4 xv[16];
        const int64_t j0 = int64_t(seg) * 128;
        const uint4 *xp = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(a.x) + j0);
#pragma unroll
        for (int q = 0; q < 16; ++q) xv[q] = (j0 + 8 * q < a.d_in) ? xp[q] : make_uint4(0, 0, 0, 0);
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
        constexpr int SEGC = 128 / D;
        const int nmine = (nrows > slot) ? (nrows - slot + rs - 1) / rs : 0;
        const int64_t base = (row_begin + slot) * a.pitch + int64_t(seg) * SEGC;
        const int64_t step = int64_t(rs) * a.pitch;
        RowData<D, S> r0, r1;
        if (nmine > 0) load_row<D, S>(r0, M, base);
        int i = 0;
        for (; i + 1 < nmine; i += 2) {
            load_row<D, S>(r1, M, base + int64_t(i + 1) * step);
            s_red[(slot + i * rs) * nseg + seg] = row_dot<D, S>(r0, xv, s_tab, M);
            if (i + 2 < nmine) load_row<D, S>(r0, M, base + int64_t(i + 2) * step);
            s_red[(slot + (i + 1) * rs) * nseg + seg] = row_dot<D, S>(r1, xv, s_tab, M);
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
        const int8_t *q8r = M.q8 + row * a.k;
        for (int64_t p = g; p < a.k; p += G) v = __builtin_fmaf(float(q8r[p]), s_xs[p], v);
        for (int q = g; q < M.rank; q += G) v = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], v);
        for (int o = G >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
        if (g == 0) {
            if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(v);
            else static_cast<float *>(M.y)[row] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 activations: the fp32 decoder table and fp32 arithmetic throughout.
// One wave per row, lanes stride over the chunks.
// ---------------------------------------------------------------------------
template <int D, int S>
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
    const float *x = static_cast<const float *>(a.x);
    const int64_t C = a.d_in / D;
    float acc = 0.0f;
    for (int64_t c = lane; c < C; c += 64) {
        float xv[D];
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int64_t col = c * D + j;
            xv[j] = (a.k > 0 && is_protected(M.idx, a.k, col)) ? 0.0f : x[col];
        }
        const int64_t off = row * a.pitch + c;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint32_t code = (D == 8) ? uint32_t(static_cast<const uint8_t *>(M.codes[s])[off])
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
        acc = __builtin_fmaf(float(M.q8[row * a.k + p]), M.scale[p] * x[M.idx[p]], acc);
    for (int q = lane; q < M.rank; q += 64) acc = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], acc);
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) {
        if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(acc);
        else static_cast<float *>(M.y)[row] = acc;
    }
}

template <int D>
hipError_t launch_f32(int stages, const GemvArgs &a, int64_t rows, hipStream_t st)
{
    const dim3 grid(unsigned((rows + 3) / 4));
    switch (stages) {
    case 1: hipLaunchKernelGGL((gemv_f32_kernel<D, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((gemv_f32_kernel<D, 2>), grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL((gemv_f32_kernel<D, 3>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((gemv_f32_kernel<D, 4>), grid, dim3(256), 0, st, a); break;
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

GemvArgs make_args(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                   const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype, void *ws)
{
    GemvArgs a{};
    a.n = n;
    a.d_in = layers[0].d_in;
    a.pitch = layers[0].pitch;
    a.k = layers[0].k;
    a.x = x;
    a.x_bf16 = (x_dtype == BSQ_BF16);
    a.y_bf16 = (y_dtype == BSQ_BF16);
    float *wt = static_cast<float *>(ws);
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
            }
        }
        M.idx = L.prot_idx;
        M.q8 = L.prot_q8;
        M.scale = L.prot_scale;
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

size_t gemv_ws_bytes(const bsq_config &cfg, int64_t n, int64_t d_in)
{
    (void)cfg;
    (void)d_in;
    return align256(size_t(n) * BSQ_MAX_LORA_RANK * 4);
}

size_t gemv_stream_lds_bytes(const bsq_config &cfg, int64_t d_in, int64_t nseg_rpb)
{
    const int64_t words = (d_in + 31) / 32;
    const int64_t k = cfg.protect_num ? (d_in * cfg.protect_num + cfg.protect_den - 1) / cfg.protect_den : 0;
    return ((cfg.d == 8) ? size_t(cfg.stages) * 256 * 16 : 0) + size_t(nseg_rpb) * 4 +
           size_t((words + 3) & ~int64_t(3)) * 4 + size_t(k) * 4;
}

hipError_t launch_gemv_prep(const bsq_config &cfg, int n, const bsq_layer *layers, const bsq_lora *loras,
                            const void *x, int x_dtype, void *ws, hipStream_t st)
{
    bool any = false;
    for (int m = 0; m < n && loras; ++m) any |= (loras[m].rank > 0);
    if (!any) return hipSuccess;
    const GemvArgs a = make_args(cfg, n, nullptr, layers, loras, x, x_dtype, nullptr, BSQ_F32, ws);
    hipLaunchKernelGGL(gemv_lora_prep_kernel, dim3(unsigned(n * BSQ_MAX_LORA_RANK)), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_gemv_run(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                           const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype,
                           void *ws, hipStream_t st)
{
    const int D = cfg.d, S = cfg.stages;
    GemvArgs a = make_args(cfg, n, codecs, layers, loras, x, x_dtype, y, y_dtype, ws);
    int64_t rows_total = 0;
    for (int m = 0; m < n; ++m) rows_total += layers[m].d_out;
    if (rows_total == 0) return hipSuccess;
    if (x_dtype != BSQ_BF16)
        return (D == 8) ? launch_f32<8>(S, a, rows_total, st) : launch_f32<16>(S, a, rows_total, st);

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
    return (D == 8) ? launch_stream<8>(S, a, nt, int(blocks), shm, st)
                    : launch_stream<16>(S, a, nt, int(blocks), shm, st);
}

}  // namespace bsq
