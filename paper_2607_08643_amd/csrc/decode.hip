// Decoder assembly (eq. parallel_stage_decode and eq. protected_8bit_scatter):
// every stage is decoded independently from its code plane and the stage
// terms are summed (the stage index is folded into each thread's work, so the
// stages decode in parallel rather than one after the other); the protected
// columns are then taken from the int8 payload. The stage sum is the fmaf
// chain of the definition, so the fp32 output is bit-identical to it.
#include <type_traits>

#include "bsq_internal.h"

namespace bsq {
namespace {

struct DecodeArgs {
    int64_t d_out, d_in, pitch, C, k, words;
    const void *codes[BSQ_MAX_STAGES];
    const uint16_t *gains[BSQ_MAX_STAGES];
    const float *tab32[BSQ_MAX_STAGES];
    const int32_t *idx;
    const int8_t *q8;
    const float *scale;
    void *out;
    int pfmt;        // bsq_prot_format of q8
    int accumulate;  // start each element from the fp32 value already in out (sequential stages)
    int scatter;     // write the protected columns (the last stage of a sequential decode)
};

// A block walks the tiles of one matrix (grid-stride, so the decoder tables
// and the protected-column metadata are set up once per block). The four
// threads 4 r .. 4 r + 3 share row r of the tile: each loads the row's 16
// codes and gains of every stage (the four lanes read the same words) and
// assembles chunks t % 4 + 4 u, u = 0 .. 3, so that at each u the four lanes
// write adjacent chunks (64 contiguous bytes of W_hat per row at d = 8 bf16)
// and every store instruction of a wave fills whole runs. Tiles always lie
// inside the padded planes, so the loads of the next tile are issued
// unconditionally while the current one is assembled; only the stores check
// the row and chunk bounds.
//
// Protected columns: the position p of column j in the ascending index list
// is the number of protected columns before it, i.e. the rank of the first
// protected column of j's 32-column word plus the set bits of that word
// below j (both kept in LDS), so no search over the list is needed.
// D outputs per chunk, B code bits per stage (B = D unless the codec has a
// linear encoder); the fp32 tables are in LDS for D = B = 8.
template <int D, int B, int S, bool BF16OUT>
__global__ __launch_bounds__(256) void decode_kernel(DecodeArgs a)
{
    constexpr bool TAB_LDS = (D == 8 && B == 8);
    extern __shared__ uint32_t s_mem[];
    // [words4] protected bitmap, [words4] rank of each word's first protected
    // column, [k4] scales, then (D = B = 8) the fp32 tables
    const int64_t words4 = (a.words + 3) & ~int64_t(3), k4 = (a.k + 3) & ~int64_t(3);
    uint32_t *s_bits = s_mem;
    int32_t *s_rank = reinterpret_cast<int32_t *>(s_mem + words4);
    float *s_scale = reinterpret_cast<float *>(s_mem + 2 * words4);
    float *s_tab = reinterpret_cast<float *>(s_mem + 2 * words4 + k4);
    const int64_t m = blockIdx.y;
    const int t = threadIdx.x;
    const int32_t *idx = a.idx ? a.idx + m * a.k : nullptr;
    if (a.k > 0) {
        for (int64_t w = t; w < a.words; w += blockDim.x) s_bits[w] = 0u;
        __syncthreads();
        for (int64_t p = t; p < a.k; p += blockDim.x) {
            const int32_t j = idx[p];
            s_scale[p] = a.scale[m * a.k + p];
            if (j >= 0 && j < a.d_in) {
                atomicOr(&s_bits[j >> 5], 1u << (j & 31));
                const int32_t jp = (p > 0) ? idx[p - 1] : -1;
                if (jp < 0 || (jp >> 5) != (j >> 5)) s_rank[j >> 5] = int32_t(p);
            }
        }
    }
    if constexpr (TAB_LDS) {
        // entry c of stage s: floats 0-3 at float4 (s 512 + c), 4-7 at
        // (s 512 + 256 + c): the two 16-byte reads of a wave spread over the
        // banks by the code
        for (int e = t; e < S * 256 * 8; e += blockDim.x) {
            const int s = e / (256 * 8), r = e - s * 256 * 8, code = r >> 3, f = r & 7;
            s_tab[((s * 512 + (f >> 2) * 256 + code) << 2) + (f & 3)] = a.tab32[s][r];
        }
    }
    __syncthreads();

    const int64_t nb = a.pitch / 16;                 // tiles per 64-row group
    const int64_t tiles = (a.d_out + 63) / 64 * nb;  // tiles of this matrix
    const int64_t kp = q8_pitch(a.k);
    const int r = t >> 2, cl = t & 3;  // row within the tile, first chunk (chunks cl + 4 u)
    const int64_t pbase = m * plane_elems(a.d_out, a.pitch) + 16 * r;

    // the row's 16 codes (B / 8 16-byte words) and 16 gains (two words) per stage
    uint4 code[2][S][B / 8];
    uint4 gain[2][S][2];
    auto load = [&](int P, int64_t tile) {
        const int64_t e = pbase + tile * 1024;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint4 *cp = reinterpret_cast<const uint4 *>(static_cast<const uint8_t *>(a.codes[s]) + e * (B / 8));
#pragma unroll
            for (int h = 0; h < B / 8; ++h) code[P][s][h] = cp[h];
            const uint4 *gp = reinterpret_cast<const uint4 *>(a.gains[s] + e);
            gain[P][s][0] = gp[0];
            gain[P][s][1] = gp[1];
        }
    };
    // 32-bit word w of a 16-byte word
    auto word = [](const uint4 &v, int w) { return (w == 0) ? v.x : (w == 1) ? v.y : (w == 2) ? v.z : v.w; };
    auto body = [&](int P, int64_t tile) {
        const int64_t rg = tile / nb, cb = tile - rg * nb;
        const int64_t i = rg * 64 + r;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int cc = cl + 4 * u;  // chunk within the tile's row
            const int64_t c = cb * 16 + cc;
            const int64_t o = (m * a.d_out + i) * a.d_in + c * D;
            const bool live = i < a.d_out && c < a.C;
            float v[D];
#pragma unroll
            for (int j = 0; j < D; ++j) v[j] = 0.0f;
            if constexpr (!BF16OUT) {
                if (a.accumulate && live) {  // the running stage sum of the earlier launches
                    const float4 *src = reinterpret_cast<const float4 *>(static_cast<const float *>(a.out) + o);
#pragma unroll
                    for (int q = 0; q < D / 4; ++q) {
                        const float4 w4 = src[q];
                        v[4 * q + 0] = w4.x;
                        v[4 * q + 1] = w4.y;
                        v[4 * q + 2] = w4.z;
                        v[4 * q + 3] = w4.w;
                    }
                }
            }
#pragma unroll
            for (int s = 0; s < S; ++s) {
                uint32_t cw;
                if constexpr (B == 8) cw = (word(code[P][s][0], cc >> 2) >> (8 * (cc & 3))) & 0xffu;
                else cw = (word(code[P][s][cc >> 3], (cc >> 1) & 3) >> (16 * (cc & 1))) & 0xffffu;
                const uint32_t gw = word(gain[P][s][cc >> 3], (cc >> 1) & 3);
                const float g = f16_bits_to_f32(uint16_t(gw >> (16 * (cc & 1))));
#pragma unroll
                for (int q = 0; q < D / 4; ++q) {
                    const float4 tv = TAB_LDS ? reinterpret_cast<const float4 *>(s_tab)[s * 512 + q * 256 + cw]
                                              : reinterpret_cast<const float4 *>(a.tab32[s] + size_t(cw) * D)[q];
                    v[4 * q + 0] = __builtin_fmaf(g, tv.x, v[4 * q + 0]);
                    v[4 * q + 1] = __builtin_fmaf(g, tv.y, v[4 * q + 1]);
                    v[4 * q + 2] = __builtin_fmaf(g, tv.z, v[4 * q + 2]);
                    v[4 * q + 3] = __builtin_fmaf(g, tv.w, v[4 * q + 3]);
                }
            }
            if (!live) continue;
            if (a.k > 0 && a.scatter) {
                const int64_t col0 = c * D;
                const uint32_t word = s_bits[col0 >> 5];
                const uint32_t pm = (word >> (col0 & 31)) & ((1u << D) - 1u);
                if (pm) {
#pragma unroll
                    for (int j = 0; j < D; ++j) {
                        if (!((pm >> j) & 1u)) continue;
                        const int b = int((col0 + j) & 31);
                        int64_t p = s_rank[col0 >> 5] + __builtin_popcount(word & ((1u << b) - 1u));
                        p = (p < 0) ? 0 : (p < a.k) ? p : a.k - 1;  // an index list that is not ascending stays in bounds
                        v[j] = payload_to_f32(uint8_t(a.q8[(m * a.d_out + i) * kp + p]), a.pfmt) * s_scale[p];
                    }
                }
            }
            if constexpr (BF16OUT) {
                uint32_t h[D / 2];
#pragma unroll
                for (int j = 0; j < D / 2; ++j) h[j] = uint32_t(f32_to_bf16(v[2 * j])) | (uint32_t(f32_to_bf16(v[2 * j + 1])) << 16);
                uint4 *dst = reinterpret_cast<uint4 *>(static_cast<uint16_t *>(a.out) + o);
#pragma unroll
                for (int q = 0; q < D / 8; ++q) dst[q] = make_uint4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
            } else {
                float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(a.out) + o);
#pragma unroll
                for (int q = 0; q < D / 4; ++q)
                    dst[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
            }
        }
    };
    int64_t tile = blockIdx.x;
    if (tile >= tiles) return;
    load(0, tile);
    for (;;) {
        const int64_t t1 = tile + gridDim.x;
        load(1, (t1 < tiles) ? t1 : tile);
        body(0, tile);
        if (t1 >= tiles) break;
        const int64_t t2 = t1 + gridDim.x;
        load(0, (t2 < tiles) ? t2 : t1);
        body(1, t1);
        if (t2 >= tiles) break;
        tile = t2;
    }
}

template <int D, int B, bool BF16OUT>
hipError_t launch_decode_t(int stages, const DecodeArgs &a, int64_t n_mats, hipStream_t st)
{
    const int64_t tiles = (a.d_out + 63) / 64 * (a.pitch / 16);
    if (tiles == 0 || n_mats == 0) return hipSuccess;
    // about eight blocks per CU in all, each walking its share of the tiles
    int64_t gx = (2048 + n_mats - 1) / n_mats;
    if (gx > tiles) gx = tiles;
    if (gx < 1) gx = 1;
    const dim3 grid = dim3(unsigned(gx), unsigned(n_mats));
    const size_t shm = size_t((a.words + 3) & ~int64_t(3)) * 8 + size_t((a.k + 3) & ~int64_t(3)) * 4 +
                       ((D == 8 && B == 8) ? size_t(stages) * 256 * 8 * 4 : 0);
    switch (stages) {
    case 1: hipLaunchKernelGGL((decode_kernel<D, B, 1, BF16OUT>), grid, dim3(256), shm, st, a); break;
    case 2: hipLaunchKernelGGL((decode_kernel<D, B, 2, BF16OUT>), grid, dim3(256), shm, st, a); break;
    case 3: hipLaunchKernelGGL((decode_kernel<D, B, 3, BF16OUT>), grid, dim3(256), shm, st, a); break;
    default: hipLaunchKernelGGL((decode_kernel<D, B, 4, BF16OUT>), grid, dim3(256), shm, st, a); break;
    }
    return hipGetLastError();
}

// the (d, b) instantiation for a configuration
template <bool BF16OUT>
hipError_t launch_decode_db(const bsq_config &cfg, int stages, const DecodeArgs &a, int64_t n_mats, hipStream_t st)
{
    if (cfg.d == 8) return (cfg.b == 8) ? launch_decode_t<8, 8, BF16OUT>(stages, a, n_mats, st)
                                        : launch_decode_t<8, 16, BF16OUT>(stages, a, n_mats, st);
    return (cfg.b == 16) ? launch_decode_t<16, 16, BF16OUT>(stages, a, n_mats, st)
                         : launch_decode_t<16, 8, BF16OUT>(stages, a, n_mats, st);
}

}  // namespace

hipError_t launch_decode(const bsq_config &cfg, const void *codec, const bsq_layer &L, void *w_hat,
                         int out_dtype, hipStream_t st)
{
    DecodeArgs a{};
    a.d_out = L.d_out;
    a.d_in = L.d_in;
    a.pitch = L.pitch;
    a.C = L.d_in / cfg.d;
    a.k = L.k;
    a.words = (L.k > 0) ? (L.d_in + 31) / 32 : 0;
    const char *cb = static_cast<const char *>(codec);
    for (int s = 0; s < cfg.stages; ++s) {
        a.codes[s] = L.codes[s];
        a.gains[s] = L.gains[s];
        a.tab32[s] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, s));
    }
    a.idx = L.prot_idx;
    a.q8 = L.prot_q8;
    a.scale = L.prot_scale;
    a.out = w_hat;
    a.pfmt = cfg.protect_format;
    a.scatter = 1;
    return (out_dtype == BSQ_BF16) ? launch_decode_db<true>(cfg, cfg.stages, a, L.n_mats, st)
                                   : launch_decode_db<false>(cfg, cfg.stages, a, L.n_mats, st);
}

// One residual stage of a sequential decode: W_hat = fmaf(gain, D_s(code),
// W_hat or 0) over the stage's plane, the protected columns written with the
// last stage. Called for s = 0 .. S-1 (accumulating from s = 1) it gives the
// bits of the stage-parallel decode, one launch and one fp32 round trip of
// W_hat per stage.
hipError_t launch_decode_stage(const bsq_config &cfg, const void *codec, const bsq_layer &L, int stage,
                               int accumulate, void *w_hat, hipStream_t st)
{
    DecodeArgs a{};
    a.d_out = L.d_out;
    a.d_in = L.d_in;
    a.pitch = L.pitch;
    a.C = L.d_in / cfg.d;
    a.k = L.k;
    a.words = (L.k > 0) ? (L.d_in + 31) / 32 : 0;
    const char *cb = static_cast<const char *>(codec);
    a.codes[0] = L.codes[stage];
    a.gains[0] = L.gains[stage];
    a.tab32[0] = reinterpret_cast<const float *>(cb + codec_tab32_offset(cfg, stage));
    a.idx = L.prot_idx;
    a.q8 = L.prot_q8;
    a.scale = L.prot_scale;
    a.out = w_hat;
    a.pfmt = cfg.protect_format;
    a.accumulate = accumulate;
    a.scatter = (stage == cfg.stages - 1);
    return launch_decode_db<false>(cfg, 1, a, L.n_mats, st);
}

}  // namespace bsq
