// Fused decode-GEMV at batch 1 (the direct computation from binary spherical
// codes that Section V names as future work):
//   y_i = sum_c sum_s gain_s(i,c) * <D_s(code_s(i,c)), x~_c>
//         + sum_p q8(i,p) * (scale_p x_{idx_p}) + sum_r B(i,r) (A x)_r
// where x~ is x with the protected input columns zeroed (those columns come
// from the int8 path, eq. protected_8bit_scatter) and the stage sum is the
// parallel residual decoding of eq. parallel_stage_decode.
//
// The main kernel streams the code and gain planes once from HBM with 128-bit
// loads. A thread owns one 128-input segment of x~ (16 chunks at d = 8,
// 8 chunks at d = 16) in registers and walks down the rows with it; the
// decoded vectors come from a bf16 table (LDS at d = 8, L2 at d = 16) and are
// dotted with x~ by v_dot2_f32_bf16 with fp32 accumulation. Per-row partial
// sums are reduced through LDS, where the epilogue also adds the int8 and
// LoRA terms.
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
    int64_t tile_begin;
    void *xt;     // workspace: masked x, [pitch * d], bf16 or fp32
    float *t;     // workspace: A x, [16]
    float *xs;    // workspace: scale_p * x_{idx_p}, [k]
    void *y;
};

struct GemvArgs {
    GemvMat mat[BSQ_MAX_GROUP];
    int n;
    int64_t d_in, pitch, k, nseg, rs, total_tiles;
    const void *x;
    int x_bf16, y_bf16;
};

__device__ __forceinline__ float load_x(const void *x, int64_t j, int bf)
{
    return bf ? bf16_to_f32(static_cast<const uint16_t *>(x)[j]) : static_cast<const float *>(x)[j];
}

// ---------------------------------------------------------------------------
// Activation prep: x~ (masked, zero-padded to pitch*d), t = A x, xs.
// Block roles: [0, nxb) x~ ; [nxb, nxb + n*16) LoRA rows ; then xs.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemv_prep_kernel(const GemvArgs a, int64_t padded_len, int64_t nxb)
{
    __shared__ float red[256];
    const int64_t b = blockIdx.x;
    const int t = threadIdx.x;
    if (b < nxb) {
        // x~[m][j]: x_j for unprotected j < d_in, else 0 (padding to pitch * d)
        const int64_t e = b * 256 + t;
        const int64_t m = e / padded_len;
        const int64_t j = e - m * padded_len;
        if (m >= a.n) return;
        const GemvMat &M = a.mat[m];
        const bool keep = j < a.d_in && !(a.k > 0 && is_protected(M.idx, a.k, j));
        if (a.x_bf16)
            static_cast<uint16_t *>(M.xt)[j] = keep ? static_cast<const uint16_t *>(a.x)[j] : uint16_t(0);
        else
            static_cast<float *>(M.xt)[j] = keep ? static_cast<const float *>(a.x)[j] : 0.0f;
        return;
    }
    if (b < nxb + int64_t(a.n) * BSQ_MAX_LORA_RANK) {
        // t[m][r] = sum_j A[r][j] x_j (unmasked x)
        const int64_t m = (b - nxb) / BSQ_MAX_LORA_RANK;
        const int r = int((b - nxb) % BSQ_MAX_LORA_RANK);
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
    // xs[m][p] = scale_p * x_{idx_p}
    if (a.k == 0) return;
    const int64_t e = (b - nxb - int64_t(a.n) * BSQ_MAX_LORA_RANK) * 256 + t;
    const int64_t m = e / a.k;
    const int64_t p = e - m * a.k;
    if (m >= a.n) return;
    const GemvMat &M = a.mat[m];
    M.xs[p] = M.scale[p] * load_x(a.x, M.idx[p], a.x_bf16);
}

// ---------------------------------------------------------------------------
// Main kernel, bf16 activations.
// ---------------------------------------------------------------------------
template <int D, int S, int ITER>
__global__ __launch_bounds__(512) void gemv_bf16_kernel(const GemvArgs a)
{
    constexpr int SEGC = 128 / D;  // chunks per segment
    extern __shared__ uint4 s_mem[];
    uint4 *s_tab = s_mem;  // D == 8: [S][256] entries of 8 bf16
    float *s_red = reinterpret_cast<float *>(s_mem + ((D == 8) ? S * 256 : 0));

    const int NT = blockDim.x;
    const int t = threadIdx.x;
    const int nseg = int(a.nseg), rs = int(a.rs);
    const int slot = t / nseg, seg = t - slot * nseg;
    const bool active = slot < rs;
    const int R = rs * ITER;
    int G = 64;
    while (G > 1 && G * R > NT) G >>= 1;

    int cur = -1;
    uint4 xv[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) xv[q] = make_uint4(0, 0, 0, 0);

    for (int64_t tile = blockIdx.x; tile < a.total_tiles; tile += gridDim.x) {
        int m = 0;
        while (m + 1 < a.n && tile >= a.mat[m + 1].tile_begin) ++m;
        const GemvMat &M = a.mat[m];
        if (m != cur) {
            cur = m;
            if (active) {
                const uint4 *src = reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(M.xt) + int64_t(seg) * 128);
#pragma unroll
                for (int q = 0; q < 16; ++q) xv[q] = src[q];
            }
            if constexpr (D == 8) {
                for (int e = t; e < S * 256; e += NT) {
                    const int s = e >> 8;
                    s_tab[e] = reinterpret_cast<const uint4 *>(M.tab16[s])[e & 255];
                }
                __syncthreads();
            }
        }
        const int64_t row0 = (tile - M.tile_begin) * R;
        float part[ITER];
        uint4 cw[ITER][S];
        uint4 gw[ITER][S][2];
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int64_t row = row0 + int64_t(it) * rs + slot;
            part[it] = 0.0f;
            if (active && row < M.d_out) {
                const int64_t off = row * a.pitch + int64_t(seg) * SEGC;  // in chunks
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    if constexpr (D == 8)
                        cw[it][s] = *reinterpret_cast<const uint4 *>(static_cast<const uint8_t *>(M.codes[s]) + off);
                    else
                        cw[it][s] = *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(M.codes[s]) + off);
                    const uint4 *gp = reinterpret_cast<const uint4 *>(M.gains[s] + off);
                    gw[it][s][0] = gp[0];
                    if constexpr (D == 8) gw[it][s][1] = gp[1];
                }
            }
        }
#pragma unroll
        for (int it = 0; it < ITER; ++it) {
            const int64_t row = row0 + int64_t(it) * rs + slot;
            if (!(active && row < M.d_out)) continue;
            float acc = 0.0f;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const uint32_t *cws = reinterpret_cast<const uint32_t *>(&cw[it][s]);
                const uint32_t *gws = reinterpret_cast<const uint32_t *>(&gw[it][s][0]);
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
            part[it] = acc;
        }
        // reduce the segment partials of each row, add the int8 and LoRA terms
#pragma unroll
        for (int it = 0; it < ITER; ++it) s_red[it * NT + t] = part[it];
        __syncthreads();
        for (int r = t / G; r < R; r += NT / G) {
            const int g = t & (G - 1);
            const int it = r / rs, sl = r - it * rs;
            const int64_t row = row0 + int64_t(it) * rs + sl;
            float v = 0.0f;
            if (row < M.d_out) {
                const float *rp = s_red + it * NT + sl * nseg;
                for (int q = g; q < nseg; q += G) v += rp[q];
                for (int64_t p = g; p < a.k; p += G) v = __builtin_fmaf(float(M.q8[row * a.k + p]), M.xs[p], v);
                for (int q = g; q < M.rank; q += G)
                    v = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], v);
            }
            for (int o = G >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
            if (g == 0 && row < M.d_out) {
                if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(v);
                else static_cast<float *>(M.y)[row] = v;
            }
        }
        __syncthreads();
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
    // waves enumerate (matrix, row) pairs in order
    int m = 0;
    int64_t row = wave;
    while (m < a.n && row >= a.mat[m].d_out) {
        row -= a.mat[m].d_out;
        ++m;
    }
    if (m >= a.n) return;
    const GemvMat &M = a.mat[m];
    const float *xt = static_cast<const float *>(M.xt);
    const int64_t C = a.d_in / D;
    float acc = 0.0f;
    for (int64_t c = lane; c < C; c += 64) {
        const int64_t off = row * a.pitch + c;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint32_t code = (D == 8) ? uint32_t(static_cast<const uint8_t *>(M.codes[s])[off])
                                           : uint32_t(static_cast<const uint16_t *>(M.codes[s])[off]);
            const float g = f16_bits_to_f32(M.gains[s][off]);
            const float *y = M.tab32[s] + size_t(code) * D;
            float dsum = 0.0f;
#pragma unroll
            for (int j = 0; j < D; ++j) dsum = __builtin_fmaf(y[j], xt[c * D + j], dsum);
            acc = __builtin_fmaf(g, dsum, acc);
        }
    }
    for (int64_t p = lane; p < a.k; p += 64) acc = __builtin_fmaf(float(M.q8[row * a.k + p]), M.xs[p], acc);
    for (int q = lane; q < M.rank; q += 64) acc = __builtin_fmaf(bf16_to_f32(M.B[row * M.rank + q]), M.t[q], acc);
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) {
        if (a.y_bf16) static_cast<uint16_t *>(M.y)[row] = f32_to_bf16(acc);
        else static_cast<float *>(M.y)[row] = acc;
    }
}

template <int D, int S>
hipError_t launch_main_bf16(const GemvArgs &a, int nt, int iter, int grid, hipStream_t st)
{
    const size_t shm = ((D == 8) ? size_t(S) * 256 * 16 : 0) + size_t(iter) * nt * 4;
    switch (iter) {
    case 1: hipLaunchKernelGGL((gemv_bf16_kernel<D, S, 1>), dim3(grid), dim3(nt), shm, st, a); break;
    case 2: hipLaunchKernelGGL((gemv_bf16_kernel<D, S, 2>), dim3(grid), dim3(nt), shm, st, a); break;
    default: hipLaunchKernelGGL((gemv_bf16_kernel<D, S, 4>), dim3(grid), dim3(nt), shm, st, a); break;
    }
    return hipGetLastError();
}

template <int D>
hipError_t launch_main_f32(int stages, const GemvArgs &a, int64_t rows, hipStream_t st)
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

struct WsParts {
    size_t xt, t, xs, per;
};
WsParts ws_parts(const bsq_config &cfg, int64_t d_in)
{
    const int64_t C = d_in / cfg.d;
    const int64_t pitch = (C + BSQ_PITCH_ALIGN - 1) / BSQ_PITCH_ALIGN * BSQ_PITCH_ALIGN;
    const int64_t k = cfg.protect_num ? (d_in * cfg.protect_num + cfg.protect_den - 1) / cfg.protect_den : 0;
    WsParts w;
    w.xt = align256(size_t(pitch) * cfg.d * 4);
    w.t = align256(BSQ_MAX_LORA_RANK * 4);
    w.xs = align256(size_t(k > 0 ? k : 1) * 4);
    w.per = w.xt + w.t + w.xs;
    return w;
}

}  // namespace

size_t gemv_ws_bytes(const bsq_config &cfg, int64_t n, int64_t d_in) { return size_t(n) * ws_parts(cfg, d_in).per; }

hipError_t launch_gemv(const bsq_config &cfg, int n, const void *const *codecs, const bsq_layer *layers,
                       const bsq_lora *loras, const void *x, int x_dtype, void *const *y, int y_dtype, void *ws,
                       hipStream_t st)
{
    const int D = cfg.d, S = cfg.stages;
    const int64_t d_in = layers[0].d_in;
    const int64_t pitch = layers[0].pitch;
    const bool xbf = (x_dtype == BSQ_BF16);
    GemvArgs a{};
    a.n = n;
    a.d_in = d_in;
    a.pitch = pitch;
    a.k = layers[0].k;
    a.x = x;
    a.x_bf16 = xbf;
    a.y_bf16 = (y_dtype == BSQ_BF16);
    const WsParts wp = ws_parts(cfg, d_in);
    char *wb = static_cast<char *>(ws);
    int64_t rows_total = 0;
    for (int m = 0; m < n; ++m) {
        GemvMat &M = a.mat[m];
        const bsq_layer &L = layers[m];
        const char *cb = static_cast<const char *>(codecs[m]);
        for (int s = 0; s < S; ++s) {
            M.codes[s] = L.codes[s];
            M.gains[s] = L.gains[s];
            M.tab16[s] = reinterpret_cast<const uint16_t *>(cb + codec_tab16_offset(cfg, s));
            M.tab32[s] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, s));
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
        M.y = y[m];
        M.xt = wb + m * wp.per;
        M.t = reinterpret_cast<float *>(wb + m * wp.per + wp.xt);
        M.xs = reinterpret_cast<float *>(wb + m * wp.per + wp.xt + wp.t);
        rows_total += L.d_out;
    }
    // prep: x~ for every matrix, LoRA t rows, xs
    const int64_t padded = pitch * D;
    const int64_t nxb = (n * padded + 255) / 256;
    const int64_t nsb = (a.k > 0) ? (n * a.k + 255) / 256 : 0;
    hipLaunchKernelGGL(gemv_prep_kernel, dim3(unsigned(nxb + n * BSQ_MAX_LORA_RANK + nsb)), dim3(256), 0, st, a,
                       padded, nxb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || rows_total == 0) return e;

    if (!xbf) {
        return (D == 8) ? launch_main_f32<8>(S, a, rows_total, st) : launch_main_f32<16>(S, a, rows_total, st);
    }
    const int SEGC = 128 / D;
    const int64_t nseg = pitch / SEGC;
    // block size: the multiple of 64 in {256, 512} that leaves the fewest idle threads
    int nt = 256;
    {
        double best = -1.0;
        for (int cand : {256, 512}) {
            if (nseg > cand) continue;
            const int64_t rs = cand / nseg;
            const double use = double(rs * nseg) / cand;
            if (use > best + 1e-9) {
                best = use;
                nt = cand;
            }
        }
    }
    a.nseg = nseg;
    a.rs = nt / nseg;
    int iter = 2;
    int64_t tiles = 0;
    for (int m = 0; m < n; ++m) tiles += (layers[m].d_out + a.rs * iter - 1) / (a.rs * iter);
    if (tiles < 1024) iter = 1;
    tiles = 0;
    for (int m = 0; m < n; ++m) {
        a.mat[m].tile_begin = tiles;
        tiles += (layers[m].d_out + a.rs * iter - 1) / (a.rs * iter);
    }
    a.total_tiles = tiles;
    const int grid = int(tiles < 2048 ? tiles : 2048);
    switch (S) {
    case 1: return (D == 8) ? launch_main_bf16<8, 1>(a, nt, iter, grid, st) : launch_main_bf16<16, 1>(a, nt, iter, grid, st);
    case 2: return (D == 8) ? launch_main_bf16<8, 2>(a, nt, iter, grid, st) : launch_main_bf16<16, 2>(a, nt, iter, grid, st);
    case 3: return (D == 8) ? launch_main_bf16<8, 3>(a, nt, iter, grid, st) : launch_main_bf16<16, 3>(a, nt, iter, grid, st);
    default: return (D == 8) ? launch_main_bf16<8, 4>(a, nt, iter, grid, st) : launch_main_bf16<16, 4>(a, nt, iter, grid, st);
    }
}

}  // namespace bsq
