// Encoder (Sections III-C to III-E): protected-channel scores and TopK, int8
// quantisation of the protected columns, then per chunk and stage the sign
// code, the decoded vector, the least-squares fp16 gain and the residual.
//
// Every floating-point step follows the canonical order of the definition
// (fp64 sequential column sums; fmaf chains in element order; IEEE division;
// round-to-nearest-even fp16), so codes, gains, indices and the int8 payload
// are bit-identical to it. A stack of n_mats matrices of one category is
// encoded by the same launches (the category-batched layout of Section III-G),
// which also gives the sequential column sums enough parallelism.
#include <type_traits>

#include "bsq_internal.h"

namespace bsq {
namespace {

constexpr int TOPK_THREADS = 1024;

// ---------------------------------------------------------------------------
// Column energy key_j = g_j^2 * sum_i w_ij^2 (fp64, rows in order) and the
// column absmax for Q8. One lane per column: adjacent lanes read adjacent
// columns of a row, so every row read is coalesced.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ float load_elem(const T *p);
template <>
__device__ __forceinline__ float load_elem<float>(const float *p) { return *p; }
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t *p) { return bf16_to_f32(*p); }

template <typename T>
__global__ __launch_bounds__(256) void colscore_kernel(const T *__restrict__ W, int64_t d_out, int64_t d_in,
                                                       const float *__restrict__ g, double *__restrict__ keys,
                                                       float *__restrict__ absmax, int32_t *err)
{
    const int64_t m = blockIdx.y;
    const int64_t col = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (col >= d_in) return;
    const T *p = W + m * d_out * d_in + col;
    double s = 0.0;
    float mx = 0.0f;
    // rows in order, U at a time, the next U already in flight (two register
    // buffers, branch-free steady state so the loads are not waited on early)
    constexpr int U = 32;
    float va[U], vb[U];
    auto take = [&](const float (&v)[U]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const double dv = double(v[u]);
            s = s + dv * dv;
            const float a = __builtin_fabsf(v[u]);
            if (a > mx) mx = a;
        }
    };
    int64_t i = 0;
    if (d_out >= 2 * U) {
#pragma unroll
        for (int u = 0; u < U; ++u) va[u] = load_elem<T>(p + int64_t(u) * d_in);
        for (; i + 3 * U <= d_out; i += 2 * U) {
#pragma unroll
            for (int u = 0; u < U; ++u) vb[u] = load_elem<T>(p + (i + U + u) * d_in);
            take(va);
#pragma unroll
            for (int u = 0; u < U; ++u) va[u] = load_elem<T>(p + (i + 2 * U + u) * d_in);
            take(vb);
        }
        // rows [i, i + U) are in va; the rest is done one by one below
        take(va);
        i += U;
    }
    for (; i < d_out; ++i) {
        const float v = load_elem<T>(p + i * d_in);
        const double dv = double(v);
        s = s + dv * dv;
        const float a = __builtin_fabsf(v);
        if (a > mx) mx = a;
    }
    if (g) {
        double gj = double(g[m * d_in + col]);
        s = (gj * gj) * s;
    }
    keys[m * d_in + col] = s;
    absmax[m * d_in + col] = mx;
    // a NaN or Inf makes the fp64 sum non-finite (squares of finite fp32
    // values cannot overflow it)
    if (err && !__builtin_isfinite(s)) atomicOr(err, int32_t(BSQ_DEVERR_NONFINITE));
}

// ---------------------------------------------------------------------------
// Row energy key_i = g_i^2 * sum_j w_ij^2 (fp64, columns in order) and the
// row absmax: the output-channel score, and the gate/up terms of the coupled
// MLP score. One lane per row, walking its row in 16-byte pieces (a lane
// reuses each cache line over its next loads).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void rowscore_kernel(const T *__restrict__ W, int64_t n_rows, int64_t n_cols,
                                                       const float *__restrict__ g, double *__restrict__ keys,
                                                       float *__restrict__ absmax, int32_t *err)
{
    const int64_t m = blockIdx.y;
    const int64_t row = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (row >= n_rows) return;
    const T *p = W + (m * n_rows + row) * n_cols;
    double s = 0.0;
    float mx = 0.0f;
    auto take = [&](float v) {
        const double dv = double(v);
        s = s + dv * dv;
        const float a = __builtin_fabsf(v);
        if (a > mx) mx = a;
    };
    constexpr int V = 16 / int(sizeof(T));
    const int64_t nv = n_cols / V;  // whole 16-byte pieces (rows are 16-byte aligned when n_cols % V == 0)
    if (n_cols % V == 0) {
        for (int64_t v = 0; v < nv; ++v) {
            const uint4 raw = reinterpret_cast<const uint4 *>(p)[v];
            if constexpr (sizeof(T) == 4) {
                take(__uint_as_float(raw.x));
                take(__uint_as_float(raw.y));
                take(__uint_as_float(raw.z));
                take(__uint_as_float(raw.w));
            } else {
                const uint32_t w4[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    take(bf16_to_f32(uint16_t(w4[e] & 0xffffu)));
                    take(bf16_to_f32(uint16_t(w4[e] >> 16)));
                }
            }
        }
    } else {
        for (int64_t j = 0; j < n_cols; ++j) take(load_elem<T>(p + j));
    }
    if (g) {
        const double gi = double(g[m * n_rows + row]);
        s = (gi * gi) * s;
    }
    keys[m * n_rows + row] = s;
    absmax[m * n_rows + row] = mx;
    if (err && !__builtin_isfinite(s)) atomicOr(err, int32_t(BSQ_DEVERR_NONFINITE));
}

// Coupled MLP score of channel j (eq. mlp_coupled_protection) from the three
// fp64 squared norms: |g_gate| sqrt(sg) + |g_up| sqrt(su) + |g_down| sqrt(sd),
// added left to right (correctly rounded fp64 square roots; no contraction).
__global__ __launch_bounds__(256) void coupled_score_kernel(const double *__restrict__ sg,
                                                            const double *__restrict__ su,
                                                            const double *__restrict__ sd, const float *gg,
                                                            const float *gu, const float *gd, int64_t n,
                                                            double *__restrict__ keys, double *scores)
{
    const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (j >= n) return;
    const double a = gg ? __builtin_fabs(double(gg[j])) : 1.0;
    const double b = gu ? __builtin_fabs(double(gu[j])) : 1.0;
    const double c = gd ? __builtin_fabs(double(gd[j])) : 1.0;
    const double ta = a * __builtin_sqrt(sg[j]);
    const double tb = b * __builtin_sqrt(su[j]);
    const double tc = c * __builtin_sqrt(sd[j]);
    const double v = (ta + tb) + tc;
    keys[j] = v;
    if (scores) scores[j] = v;
}

// Exclusive prefix sum over a 1024-thread block; returns the block total.
__device__ int block_exclusive_scan(int v, int *s_wave, int &total)
{
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_wave[w] = x;
    __syncthreads();
    if (t == 0) {
        int run = 0;
        for (int i = 0; i < TOPK_THREADS / 64; ++i) {
            int c = s_wave[i];
            s_wave[i] = run;
            run += c;
        }
        s_wave[TOPK_THREADS / 64] = run;
    }
    __syncthreads();
    int excl = x - v + s_wave[w];
    total = s_wave[TOPK_THREADS / 64];
    __syncthreads();
    return excl;
}

// ---------------------------------------------------------------------------
// P = TopK(key, k), ties to the lower column, stored ascending; also the
// per-column scale s_p = absmax / pmax (the payload format's largest finite
// value), the column -> p map and the bitmap of
// protected columns. One block per matrix: an MSB-first radix select over the
// 64-bit key patterns (non-negative doubles order like their bit patterns)
// finds the k-th largest key T; then all keys > T and the lowest-index keys
// equal to T are compacted in column order.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(TOPK_THREADS) void topk_kernel(const double *__restrict__ keys_all,
                                                            const float *__restrict__ absmax_all,
                                                            int64_t d_in, int64_t k, int64_t words, float pmax,
                                                            int32_t *__restrict__ idx_all,
                                                            float *__restrict__ scale_all,
                                                            int32_t *__restrict__ colmap_all,
                                                            uint32_t *__restrict__ bitmap_all)
{
    extern __shared__ uint32_t s_bits[];  // [words], the padded columns of one matrix
    __shared__ uint32_t hist[256];
    __shared__ unsigned long long s_prefix;
    __shared__ long long s_remaining, s_next_remaining;
    __shared__ int s_wave[TOPK_THREADS / 64 + 1];

    const int64_t m = blockIdx.x;
    const int t = threadIdx.x;
    const unsigned long long *keys = reinterpret_cast<const unsigned long long *>(keys_all + m * d_in);
    const float *absmax = absmax_all + m * d_in;
    int32_t *idx = idx_all + m * k;
    float *scale = scale_all + m * k;
    int32_t *colmap = colmap_all + m * d_in;
    uint32_t *bitmap = bitmap_all + m * words;

    if (t == 0) {
        s_prefix = 0ull;
        s_remaining = k;
    }
    unsigned long long mask = 0ull;
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        for (int b = t; b < 256; b += TOPK_THREADS) hist[b] = 0u;
        __syncthreads();
        const unsigned long long prefix = s_prefix;
        for (int64_t j = t; j < d_in; j += TOPK_THREADS) {
            unsigned long long u = keys[j];
            if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255ull], 1u);
        }
        __syncthreads();
        // the digit holding the rem-th largest key: with cum(dgt) the count of
        // keys in digits above dgt, the unique dgt with cum < rem <= cum + h.
        // Threads 0..255 (whole waves) own digit 255 - t; an inclusive scan
        // over those four waves gives cum + h of every digit.
        unsigned h = 0, incl = 0;
        if (t < 256) {
            h = hist[255 - t];
            incl = h;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const unsigned y = __shfl_up(incl, o, 64);
                if ((t & 63) >= o) incl += y;
            }
            if ((t & 63) == 63) s_wave[t >> 6] = int(incl);
        }
        __syncthreads();
        if (t < 256) {
            for (int w = 0; w < (t >> 6); ++w) incl += unsigned(s_wave[w]);
            const long long rem = s_remaining;
            const long long cum = (long long)(incl - h);
            if (cum < rem && rem <= (long long)incl) {
                s_prefix = prefix | (static_cast<unsigned long long>(255 - t) << shift);
                s_next_remaining = rem - cum;
            }
        }
        __syncthreads();
        if (t == 0) s_remaining = s_next_remaining;
        mask |= 255ull << shift;
        __syncthreads();
    }
    const unsigned long long T = s_prefix;
    const long long need_eq = s_remaining;

    // each thread owns a contiguous run of columns, so scans follow column order
    const int64_t per = (d_in + TOPK_THREADS - 1) / TOPK_THREADS;
    const int64_t j0 = t * per, j1 = (j0 + per < d_in) ? j0 + per : d_in;
    int n_eq = 0;
    for (int64_t j = j0; j < j1; ++j) n_eq += (keys[j] == T);
    int tot;
    int eq_rank = block_exclusive_scan(n_eq, s_wave, tot);
    int n_sel = 0;
    {
        int r = eq_rank;
        for (int64_t j = j0; j < j1; ++j) {
            unsigned long long u = keys[j];
            bool sel = (u > T) || (u == T && r < need_eq);
            if (u == T) ++r;
            n_sel += sel;
        }
    }
    int pos = block_exclusive_scan(n_sel, s_wave, tot);
    for (int64_t w = t; w < words; w += TOPK_THREADS) s_bits[w] = 0u;
    __syncthreads();
    {
        int r = eq_rank;
        for (int64_t j = j0; j < j1; ++j) {
            unsigned long long u = keys[j];
            bool sel = (u > T) || (u == T && r < need_eq);
            if (u == T) ++r;
            if (sel) {
                idx[pos] = int32_t(j);
                scale[pos] = absmax[j] / pmax;
                colmap[j] = pos;
                atomicOr(&s_bits[j >> 5], 1u << (j & 31));
                ++pos;
            } else {
                colmap[j] = -1;
            }
        }
    }
    __syncthreads();
    for (int64_t w = t; w < words; w += TOPK_THREADS) bitmap[w] = s_bits[w];
}

// ---------------------------------------------------------------------------
// A given protected column set: checks it (strictly ascending, in range),
// then writes what topk_kernel writes for a selected one: the indices, the
// scales absmax / pmax, the column -> p map and the bitmap. One block per
// matrix. An invalid entry ORs 2 into *err and is left out.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(TOPK_THREADS) void colset_kernel(const int32_t *__restrict__ idx_in,
                                                              const float *__restrict__ absmax_all, int64_t d_in,
                                                              int64_t k, int64_t words, float pmax, int32_t *idx_out,
                                                              float *__restrict__ scale_all,
                                                              int32_t *__restrict__ colmap_all,
                                                              uint32_t *__restrict__ bitmap_all, int32_t *err)
{
    extern __shared__ uint32_t s_bits[];
    const int64_t m = blockIdx.x;
    const int t = threadIdx.x;
    for (int64_t j = t; j < d_in; j += TOPK_THREADS) colmap_all[m * d_in + j] = -1;
    for (int64_t w = t; w < words; w += TOPK_THREADS) s_bits[w] = 0u;
    __syncthreads();
    for (int64_t p = t; p < k; p += TOPK_THREADS) {
        const int32_t j = idx_in[m * k + p];
        const bool ok = j >= 0 && j < d_in && (p == 0 || idx_in[m * k + p - 1] < j);
        if (!ok) {
            atomicOr(err, int32_t(BSQ_DEVERR_BAD_SET));
            continue;
        }
        colmap_all[m * d_in + j] = int32_t(p);
        atomicOr(&s_bits[j >> 5], 1u << (j & 31));
        scale_all[m * k + p] = absmax_all[m * d_in + j] / pmax;
        idx_out[m * k + p] = j;
    }
    __syncthreads();
    for (int64_t w = t; w < words; w += TOPK_THREADS) bitmap_all[m * words + w] = s_bits[w];
}

// ---------------------------------------------------------------------------
// Protected output rows (eq. protected_8bit_scatter with row slices): one
// block per (protected row p, matrix). Checks the set, then the row's absmax
// (exact in any order), scale = absmax / payload_max, the row's stored bytes
// (payload_from_f32; zero past d_in and when the scale is 0), and clears the
// row's codes and gains in every stage plane (the row is not BSQ-coded). Runs
// after the per-chunk encoder on the same stream.
// ---------------------------------------------------------------------------
struct RowProtArgs {
    const void *W;
    int64_t d_out, d_in, pitch, k;
    const int32_t *idx_in;
    int32_t *idx_out;
    int8_t *q8;       // [n_mats][k][q8_pitch(d_in)]
    float *scale;     // [n_mats][k]
    void *codes[BSQ_MAX_STAGES];
    uint16_t *gains[BSQ_MAX_STAGES];
    int stages, code_bytes, pfmt;
    int32_t *err;
};

template <typename T>
__global__ __launch_bounds__(256) void rowprot_kernel(const RowProtArgs a)
{
    __shared__ float s_max[4];
    const int64_t p = blockIdx.x, m = blockIdx.y;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int32_t i = a.idx_in[m * a.k + p];
    const bool ok = i >= 0 && i < a.d_out && (p == 0 || a.idx_in[m * a.k + p - 1] < i);
    if (!ok) {
        if (t == 0) atomicOr(a.err, int32_t(BSQ_DEVERR_BAD_SET));
        return;
    }
    const T *row = static_cast<const T *>(a.W) + (m * a.d_out + i) * a.d_in;
    float mx = 0.0f;
    for (int64_t j = t; j < a.d_in; j += 256) {
        const float v = __builtin_fabsf(load_elem<T>(row + j));
        if (v > mx) mx = v;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float y = __shfl_xor(mx, o, 64);
        mx = (y > mx) ? y : mx;
    }
    if (lane == 0) s_max[wave] = mx;
    __syncthreads();
    float am = s_max[0];
#pragma unroll
    for (int w = 1; w < 4; ++w) am = (s_max[w] > am) ? s_max[w] : am;
    const float sc = am / payload_max(a.pfmt);
    if (t == 0) {
        a.scale[m * a.k + p] = sc;
        a.idx_out[m * a.k + p] = i;
    }
    const int64_t qp = q8_pitch(a.d_in);
    int8_t *qrow = a.q8 + (m * a.k + p) * qp;
    for (int64_t j = t; j < qp; j += 256)
        qrow[j] = (j < a.d_in && sc != 0.0f) ? int8_t(payload_from_f32(load_elem<T>(row + j) / sc, a.pfmt)) : int8_t(0);
    const int64_t base = m * plane_elems(a.d_out, a.pitch);
    for (int64_t c = t; c < a.pitch; c += 256) {
        const int64_t gid = base + tile_index(i, c, a.pitch);
        for (int s = 0; s < a.stages; ++s) {
            if (a.code_bytes == 1) static_cast<uint8_t *>(a.codes[s])[gid] = 0;
            else static_cast<uint16_t *>(a.codes[s])[gid] = 0;
            a.gains[s][gid] = 0;
        }
    }
}

// ---------------------------------------------------------------------------
// Per-chunk encoder. One thread per chunk (padding chunks included, which get
// code 0 and gain +0).
// ---------------------------------------------------------------------------
struct EncodeArgs {
    const void *W;
    int64_t d_out, d_in, pitch, C, k, words, total;
    void *codes[BSQ_MAX_STAGES];
    uint16_t *gains[BSQ_MAX_STAGES];
    const float *tab32[BSQ_MAX_STAGES];
    int8_t *q8;
    const float *scale;
    const int32_t *colmap;
    const int32_t *idx;  // protected columns [n_mats][k] (the payload pass)
    const uint32_t *bitmap;
    int32_t *err;
    int pfmt;  // bsq_prot_format of q8
    const float *enc[BSQ_MAX_STAGES];  // linear encoder E [b][d] per stage, or null (identity)
};

// one element of the tiled planes (padding rows and chunks included):
// matrix m, row i, chunk c, at plane position gid. D inputs per chunk, B code
// bits; ENC: the stage code is the sign pattern of z = E r (E [B][D] in LDS,
// s_E), else of r itself (B = D). The decoder table is in LDS (s_tab) for
// D = B = 8, as [S][2][256][4] (the two halves of an entry 4 KiB apart, so
// that each 16-byte read of a wave spreads over the banks by the code), else
// read from the fp32 table in global memory. The protected columns of the
// chunk are masked out of the stages (their payload bytes are written by the
// kernel's separate payload pass).
// The raw words of one chunk and its protected-position mask, fetched ahead
// of the chunk's arithmetic (a thread's four chunks of a tile are requested
// together, so that their loads are in flight at once).
template <int D, typename T>
struct ChunkIn {
    static constexpr int NV = D * int(sizeof(T)) / 16;
    uint4 raw[NV];
    uint32_t pmw;  // the bitmap word of the chunk's columns (shifted and masked where used)
};

template <int D, typename T>
__device__ __forceinline__ void encode_fetch(const EncodeArgs &a, int64_t m, int64_t i, int64_t c, ChunkIn<D, T> &in)
{
    in.pmw = 0;
    if (c >= a.C || i >= a.d_out) return;
    const T *src = static_cast<const T *>(a.W) + (m * a.d_out + i) * a.d_in + c * D;
#pragma unroll
    for (int v = 0; v < ChunkIn<D, T>::NV; ++v) in.raw[v] = reinterpret_cast<const uint4 *>(src)[v];
    if (a.bitmap) in.pmw = a.bitmap[m * a.words + ((c * D) >> 5)];
}

template <int D, int B, int S, typename T, bool ENC>
__device__ __forceinline__ void encode_element(const EncodeArgs &a, const float *s_tab, const float *s_E,
                                               int64_t m, int64_t i, int64_t c, int64_t gid, const ChunkIn<D, T> &in)
{
    using code_t = typename std::conditional<B == 8, uint8_t, uint16_t>::type;
    constexpr bool TAB_LDS = (D == 8 && B == 8);

    if (c >= a.C || i >= a.d_out) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
            static_cast<code_t *>(a.codes[s])[gid] = 0;
            a.gains[s][gid] = 0;
        }
        return;
    }

    // the chunk
    float w[D];
    if constexpr (sizeof(T) == 4) {
        const float *f = reinterpret_cast<const float *>(in.raw);
#pragma unroll
        for (int j = 0; j < D; ++j) w[j] = f[j];
    } else {
        const uint16_t *h = reinterpret_cast<const uint16_t *>(in.raw);
#pragma unroll
        for (int j = 0; j < D; ++j) w[j] = bf16_to_f32(h[j]);
    }
    bool finite = true;
#pragma unroll
    for (int j = 0; j < D; ++j) finite &= __builtin_isfinite(w[j]);
    if (!finite) atomicOr(a.err, int32_t(BSQ_DEVERR_NONFINITE));

    // protected positions of this chunk, masked out of BSQ
    const uint32_t pm = (in.pmw >> ((c * D) & 31)) & ((1u << D) - 1u);
    float r[D];
#pragma unroll
    for (int j = 0; j < D; ++j) r[j] = ((pm >> j) & 1u) ? 0.0f : w[j];

#pragma unroll
    for (int s = 0; s < S; ++s) {
        uint32_t code = 0;
        if constexpr (ENC) {
            // z_m = sum_j E[m][j] r_j, the fmaf chain from +0 in j order
#pragma unroll
            for (int mm = 0; mm < B; ++mm) {
                float z = 0.0f;
#pragma unroll
                for (int j = 0; j < D; ++j) z = __builtin_fmaf(s_E[(s * B + mm) * D + j], r[j], z);
                code |= (z >= 0.0f ? 1u : 0u) << mm;
            }
        } else {
#pragma unroll
            for (int j = 0; j < D; ++j) code |= (r[j] >= 0.0f ? 1u : 0u) << j;
        }
        float yv[D];
        if constexpr (TAB_LDS) {
            const float4 *y4 = reinterpret_cast<const float4 *>(s_tab) + s * 512 + code;
            float4 lo = y4[0], hi = y4[256];
            yv[0] = lo.x; yv[1] = lo.y; yv[2] = lo.z; yv[3] = lo.w;
            yv[4] = hi.x; yv[5] = hi.y; yv[6] = hi.z; yv[7] = hi.w;
        } else if constexpr (D == 8) {
            const float *y = a.tab32[s] + size_t(code) * D;
            const float4 *y4 = reinterpret_cast<const float4 *>(y);
            float4 lo = y4[0], hi = y4[1];
            yv[0] = lo.x; yv[1] = lo.y; yv[2] = lo.z; yv[3] = lo.w;
            yv[4] = hi.x; yv[5] = hi.y; yv[6] = hi.z; yv[7] = hi.w;
        } else {
            const float4 *y4 = reinterpret_cast<const float4 *>(a.tab32[s] + size_t(code) * D);
#pragma unroll
            for (int v = 0; v < D / 4; ++v) {
                float4 q = y4[v];
                yv[4 * v + 0] = q.x; yv[4 * v + 1] = q.y; yv[4 * v + 2] = q.z; yv[4 * v + 3] = q.w;
            }
        }
        // protected positions take y = +0 (their r is +0): each of their terms
        // then adds an exact +0 to a sum that is never -0, and leaves r at +0,
        // the same as skipping them
#pragma unroll
        for (int j = 0; j < D; ++j) yv[j] = ((pm >> j) & 1u) ? 0.0f : yv[j];
        float num = 0.0f, den = 0.0f;
#pragma unroll
        for (int j = 0; j < D; ++j) {
            num = __builtin_fmaf(r[j], yv[j], num);
            den = __builtin_fmaf(yv[j], yv[j], den);
        }
        float alpha = (den > 0.0f) ? num / den : 0.0f;
        if (alpha != alpha) alpha = 0.0f;
        const uint16_t gh = gain_to_f16(alpha);
        const float ga = f16_bits_to_f32(gh);
#pragma unroll
        for (int j = 0; j < D; ++j) r[j] = __builtin_fmaf(-ga, yv[j], r[j]);
        static_cast<code_t *>(a.codes[s])[gid] = code_t(code);
        a.gains[s][gid] = gh;
    }
}

// A block walks whole 64-row x 16-chunk tiles (grid-stride), so the decoder
// tables (d = 8) are staged in LDS once per block, and a tile's matrix, row
// group and column block come from one scalar division per tile. Thread t
// takes elements t, t + 256, ... of the tile: a wave covers four rows of 16
// consecutive chunks, so its row reads are contiguous.
template <int D, int B, int S, typename T, bool ENC>
__global__ __launch_bounds__(256) void encode_kernel(EncodeArgs a)
{
    extern __shared__ float s_tab[];  // D = B = 8: [S][256][8]; then ENC: [S][B][D]
    constexpr bool TAB_LDS = (D == 8 && B == 8);
    float *s_E = s_tab + (TAB_LDS ? S * 256 * 8 : 0);
    if constexpr (TAB_LDS) {
        // entry c of stage s: floats 0-3 at float4 (s 512 + c), 4-7 at (s 512 + 256 + c)
        for (int e = threadIdx.x; e < S * 256 * 8; e += blockDim.x) {
            const int s = e / (256 * 8), r = e - s * 256 * 8, code = r >> 3, f = r & 7;
            s_tab[((s * 512 + (f >> 2) * 256 + code) << 2) + (f & 3)] = a.tab32[s][r];
        }
    }
    if constexpr (ENC) {
        for (int e = threadIdx.x; e < S * B * D; e += blockDim.x) {
            int s = e / (B * D), r = e - s * B * D;
            s_E[e] = a.enc[s][r];
        }
    }
    if constexpr (TAB_LDS || ENC) __syncthreads();
    const int64_t nb = a.pitch >> 4;
    const int64_t tiles_per_mat = ((a.d_out + 63) >> 6) * nb;
    const int64_t ntiles = a.total >> 10;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t m = tile / tiles_per_mat;
        const int64_t rem = tile - m * tiles_per_mat;
        const int64_t rg = rem / nb, blk = rem - rg * nb;
        ChunkIn<D, T> in[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = q * 256 + int(threadIdx.x);
            encode_fetch<D, T>(a, m, rg * 64 + (e >> 4), blk * 16 + (e & 15), in[q]);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = q * 256 + int(threadIdx.x);
            encode_element<D, B, S, T, ENC>(a, s_tab, s_E, m, rg * 64 + (e >> 4), blk * 16 + (e & 15), (tile << 10) + e,
                                            in[q]);
        }
    }
    // the payload pass: four bytes of a padded payload row per thread, each
    // byte the protected weight over its column's scale in the payload
    // format (zero past k, and where the scale is zero)
    if (a.q8 && a.k > 0) {
        const int64_t kp = q8_pitch(a.k), kp4 = kp >> 2;
        const int64_t n4 = (a.total / plane_elems(a.d_out, a.pitch)) * a.d_out * kp4;
        for (int64_t e = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; e < n4; e += int64_t(gridDim.x) * blockDim.x) {
            const int64_t mi = e / kp4, p0 = (e - mi * kp4) << 2;  // mi = m d_out + i
            const int64_t m = mi / a.d_out;
            uint32_t word = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t p = p0 + u;
                if (p >= a.k) break;
                // (a rejected given set leaves entries of the index list
                // unwritten: any index out of range reads as column 0, and
                // the call reports the set)
                int32_t col = a.idx[m * a.k + p];
                col = (col >= 0 && col < a.d_in) ? col : 0;
                const float sc = a.scale[m * a.k + p];
                const T wv = static_cast<const T *>(a.W)[mi * a.d_in + col];
                float w;
                if constexpr (sizeof(T) == 4) w = wv;
                else w = bf16_to_f32(wv);
                const uint32_t b = (sc != 0.0f) ? uint32_t(uint8_t(payload_from_f32(w / sc, a.pfmt))) : 0u;
                word |= b << (8 * u);
            }
            reinterpret_cast<uint32_t *>(a.q8)[e] = word;
        }
    }
}

template <int D, int B, typename T, bool ENC>
hipError_t launch_encode_chunks(int stages, const EncodeArgs &a, hipStream_t st)
{
    // at most about 16 blocks per CU; each walks its share of the tiles
    int64_t blocks = a.total >> 10;
    if (blocks > 4096) blocks = 4096;
    const dim3 grid = dim3(unsigned(blocks));
    const size_t shm = ((D == 8 && B == 8) ? size_t(stages) * 256 * 8 * 4 : 0) +
                       (ENC ? size_t(stages) * B * D * 4 : 0);
    switch (stages) {
    case 1: hipLaunchKernelGGL((encode_kernel<D, B, 1, T, ENC>), grid, dim3(256), shm, st, a); break;
    case 2: hipLaunchKernelGGL((encode_kernel<D, B, 2, T, ENC>), grid, dim3(256), shm, st, a); break;
    case 3: hipLaunchKernelGGL((encode_kernel<D, B, 3, T, ENC>), grid, dim3(256), shm, st, a); break;
    default: hipLaunchKernelGGL((encode_kernel<D, B, 4, T, ENC>), grid, dim3(256), shm, st, a); break;
    }
    return hipGetLastError();
}

template <typename T>
hipError_t launch_encode_cfg(const bsq_config &cfg, const EncodeArgs &a, hipStream_t st)
{
    const int S = cfg.stages;
    if (cfg.encoder == BSQ_ENC_IDENTITY)
        return (cfg.d == 8) ? launch_encode_chunks<8, 8, T, false>(S, a, st) : launch_encode_chunks<16, 16, T, false>(S, a, st);
    if (cfg.d == 8)
        return (cfg.b == 8) ? launch_encode_chunks<8, 8, T, true>(S, a, st) : launch_encode_chunks<8, 16, T, true>(S, a, st);
    return (cfg.b == 8) ? launch_encode_chunks<16, 8, T, true>(S, a, st) : launch_encode_chunks<16, 16, T, true>(S, a, st);
}

}  // namespace

size_t encode_ws_layout(const bsq_config &cfg, int64_t n_mats, int64_t d_out, int64_t d_in, char *base,
                        EncodeWs *ws)
{
    // scores, absmax and the channel map over the protected axis, and (row
    // axis) the selection's bitmap, which nothing reads
    const int64_t n = (cfg.protect_axis == 1) ? d_out : d_in;
    size_t off = 0;
    const size_t o_keys = off;
    off = align256(off + size_t(n_mats) * n * 8);
    const size_t o_abs = off;
    off = align256(off + size_t(n_mats) * n * 4);
    const size_t o_map = off;
    off = align256(off + size_t(n_mats) * n * 4);
    const size_t o_bits = off;
    if (cfg.protect_axis == 1) off = align256(off + size_t(n_mats) * ((n + 31) / 32) * 4);
    if (ws) {
        ws->keys = reinterpret_cast<double *>(base + o_keys);
        ws->absmax = reinterpret_cast<float *>(base + o_abs);
        ws->colmap = reinterpret_cast<int32_t *>(base + o_map);
        ws->bits = reinterpret_cast<uint32_t *>(base + o_bits);
    }
    return off;
}

size_t select_ws_layout(int64_t d_ffn, char *base, SelectWs *ws)
{
    const int64_t n = d_ffn;
    size_t off = 0, o[8];
    for (int e = 0; e < 4; ++e) {  // sg, su, sd, keys (fp64)
        o[e] = off;
        off = align256(off + size_t(n) * 8);
    }
    for (int e = 4; e < 7; ++e) {  // absmax, scale, colmap (4 bytes each; unused results of the TopK)
        o[e] = off;
        off = align256(off + size_t(n) * 4);
    }
    o[7] = off;  // bitmap
    off = align256(off + size_t((n + 31) / 32) * 4);
    if (ws) {
        ws->sg = reinterpret_cast<double *>(base + o[0]);
        ws->su = reinterpret_cast<double *>(base + o[1]);
        ws->sd = reinterpret_cast<double *>(base + o[2]);
        ws->keys = reinterpret_cast<double *>(base + o[3]);
        ws->absmax = reinterpret_cast<float *>(base + o[4]);
        ws->scale = reinterpret_cast<float *>(base + o[5]);
        ws->colmap = reinterpret_cast<int32_t *>(base + o[6]);
        ws->bits = reinterpret_cast<uint32_t *>(base + o[7]);
    }
    return off;
}

namespace {

template <typename T>
hipError_t launch_colscore(const void *W, int64_t n_mats, int64_t d_out, int64_t d_in, const float *g, double *keys,
                           float *absmax, int32_t *err, hipStream_t st)
{
    dim3 grid(unsigned((d_in + 255) / 256), unsigned(n_mats));
    hipLaunchKernelGGL(colscore_kernel<T>, grid, dim3(256), 0, st, static_cast<const T *>(W), d_out, d_in, g, keys,
                       absmax, err);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_rowscore(const void *W, int64_t n_mats, int64_t n_rows, int64_t n_cols, const float *g,
                           double *keys, float *absmax, int32_t *err, hipStream_t st)
{
    dim3 grid(unsigned((n_rows + 255) / 256), unsigned(n_mats));
    hipLaunchKernelGGL(rowscore_kernel<T>, grid, dim3(256), 0, st, static_cast<const T *>(W), n_rows, n_cols, g,
                       keys, absmax, err);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_encode(const bsq_config &cfg, const void *codec, const void *W, int w_dtype,
                         int64_t n_mats, int64_t d_out, int64_t d_in, const float *g, const int32_t *given,
                         const bsq_layer &out, int32_t *err, const EncodeWs &ws, hipStream_t st)
{
    const int64_t k = out.k;
    const bool rows = cfg.protect_axis == 1;
    const bool bf = w_dtype == BSQ_BF16;
    hipError_t e = hipSuccess;
    if (k > 0 && !rows) {
        // column scores (or, for a given set, only the column absmax)
        e = bf ? launch_colscore<uint16_t>(W, n_mats, d_out, d_in, given ? nullptr : g, ws.keys, ws.absmax,
                                           nullptr, st)
               : launch_colscore<float>(W, n_mats, d_out, d_in, given ? nullptr : g, ws.keys, ws.absmax, nullptr,
                                        st);
        if (e != hipSuccess) return e;
        const int64_t words = prot_words(out.pitch, cfg.d);
        if (given)
            hipLaunchKernelGGL(colset_kernel, dim3(unsigned(n_mats)), dim3(TOPK_THREADS), size_t(words) * 4, st,
                               given, ws.absmax, d_in, k, words, payload_max(cfg.protect_format), out.prot_idx,
                               out.prot_scale, ws.colmap, out.prot_bits, err);
        else
            hipLaunchKernelGGL(topk_kernel, dim3(unsigned(n_mats)), dim3(TOPK_THREADS), size_t(words) * 4, st,
                               ws.keys, ws.absmax, d_in, k, words, payload_max(cfg.protect_format), out.prot_idx,
                               out.prot_scale, ws.colmap, out.prot_bits);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (k > 0 && rows && !given) {
        // output-row scores and their TopK (indices to the layer; the scale,
        // map and bitmap the TopK also writes are recomputed or unused)
        e = bf ? launch_rowscore<uint16_t>(W, n_mats, d_out, d_in, g, ws.keys, ws.absmax, nullptr, st)
               : launch_rowscore<float>(W, n_mats, d_out, d_in, g, ws.keys, ws.absmax, nullptr, st);
        if (e != hipSuccess) return e;
        const int64_t words = (d_out + 31) / 32;
        hipLaunchKernelGGL(topk_kernel, dim3(unsigned(n_mats)), dim3(TOPK_THREADS), size_t(words) * 4, st, ws.keys,
                           ws.absmax, d_out, k, words, payload_max(cfg.protect_format), out.prot_idx, out.prot_scale,
                           ws.colmap, ws.bits);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    EncodeArgs a{};
    a.W = W;
    a.d_out = d_out;
    a.d_in = d_in;
    a.pitch = out.pitch;
    a.C = d_in / cfg.d;
    a.k = rows ? 0 : k;  // the per-chunk encoder masks protected columns only
    a.words = prot_words(out.pitch, cfg.d);
    a.total = n_mats * plane_elems(d_out, out.pitch);
    const char *cb = static_cast<const char *>(codec);
    for (int s = 0; s < cfg.stages; ++s) {
        a.codes[s] = out.codes[s];
        a.gains[s] = out.gains[s];
        a.tab32[s] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, s));
        if (cfg.encoder == BSQ_ENC_LINEAR) a.enc[s] = reinterpret_cast<const float *>(cb + codec_enc_offset(cfg, s));
    }
    a.q8 = rows ? nullptr : out.prot_q8;
    a.scale = out.prot_scale;
    a.colmap = ws.colmap;
    a.idx = out.prot_idx;
    a.bitmap = (k > 0 && !rows) ? out.prot_bits : nullptr;
    a.err = err;
    a.pfmt = cfg.protect_format;
    if (a.total > 0) {
        e = bf ? launch_encode_cfg<uint16_t>(cfg, a, st) : launch_encode_cfg<float>(cfg, a, st);
        if (e != hipSuccess) return e;
    }
    if (k > 0 && rows && d_in > 0) {
        RowProtArgs r{};
        r.W = W;
        r.d_out = d_out;
        r.d_in = d_in;
        r.pitch = out.pitch;
        r.k = k;
        r.idx_in = given ? given : out.prot_idx;
        r.idx_out = out.prot_idx;
        r.q8 = out.prot_q8;
        r.scale = out.prot_scale;
        for (int s = 0; s < cfg.stages; ++s) {
            r.codes[s] = out.codes[s];
            r.gains[s] = out.gains[s];
        }
        r.stages = cfg.stages;
        r.code_bytes = (cfg.b <= 8) ? 1 : 2;
        r.err = err;
        r.pfmt = cfg.protect_format;
        const dim3 grid{unsigned(k), unsigned(n_mats)};
        if (bf) hipLaunchKernelGGL(rowprot_kernel<uint16_t>, grid, dim3(256), 0, st, r);
        else hipLaunchKernelGGL(rowprot_kernel<float>, grid, dim3(256), 0, st, r);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_coupled_select(const void *Wg, const void *Wu, const void *Wd, int w_dtype, int64_t d_model,
                                 int64_t d_ffn, const float *gg, const float *gu, const float *gd, int64_t k,
                                 int32_t *idx, double *scores, int32_t *err, const SelectWs &ws, hipStream_t st)
{
    const bool bf = w_dtype == BSQ_BF16;
    hipError_t e;
    // squared norms: gate and up rows (over d_model), down columns (over d_model rows)
    e = bf ? launch_rowscore<uint16_t>(Wg, 1, d_ffn, d_model, nullptr, ws.sg, ws.absmax, err, st)
           : launch_rowscore<float>(Wg, 1, d_ffn, d_model, nullptr, ws.sg, ws.absmax, err, st);
    if (e != hipSuccess) return e;
    e = bf ? launch_rowscore<uint16_t>(Wu, 1, d_ffn, d_model, nullptr, ws.su, ws.absmax, err, st)
           : launch_rowscore<float>(Wu, 1, d_ffn, d_model, nullptr, ws.su, ws.absmax, err, st);
    if (e != hipSuccess) return e;
    e = bf ? launch_colscore<uint16_t>(Wd, 1, d_model, d_ffn, nullptr, ws.sd, ws.absmax, err, st)
           : launch_colscore<float>(Wd, 1, d_model, d_ffn, nullptr, ws.sd, ws.absmax, err, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(coupled_score_kernel, dim3(unsigned((d_ffn + 255) / 256)), dim3(256), 0, st, ws.sg, ws.su,
                       ws.sd, gg, gu, gd, d_ffn, ws.keys, scores);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (k == 0) return hipSuccess;
    const int64_t words = (d_ffn + 31) / 32;
    hipLaunchKernelGGL(topk_kernel, dim3(1u), dim3(TOPK_THREADS), size_t(words) * 4, st, ws.keys, ws.absmax, d_ffn, k,
                       words, 127.0f, idx, ws.scale, ws.colmap, ws.bits);
    return hipGetLastError();
}

}  // namespace bsq
