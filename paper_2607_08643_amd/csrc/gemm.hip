// Fused decode-GEMM for M tokens: Y = X W_hat^T + (X A^T) B^T.
//
// Two kernels. The prep kernel writes, per token row, X~ (X with the
// protected columns and the padding past d_in set to zero, padded to whole
// K steps and token tiles), the gathered protected activations X[:, idx]
// and, with LoRA, T = X A^T (fp32).
//
// The main kernel gives each block BN = 64 NT weight rows and BM = 16 MT
// tokens. Wave w owns NT groups of 16 rows; each lane decodes its B
// fragments of v_mfma_f32_16x16x32_bf16 straight from the code and gain
// planes into registers (stage terms summed by the fmaf chain of the decoder
// assembly over the fp16 gains and the fp16 decoder tables, then rounded to
// bf16), so the weight tile never goes through LDS.
// The inputs of one K step (128) are permuted identically on both operands so
// that a lane's fragments are whole chunks: MFMA input group g = lane / 16 and
// fragment q cover inputs 32 g + 8 q .. + 8 of the step. X~ tiles reach LDS
// through registers into two LDS slots (loaded two steps ahead, stored one
// step ahead), the code and gain words two steps ahead in registers; one
// barrier per step. The protected term X[:, idx] (q8 s)^T and LoRA are added in the
// epilogue; the protected products go through the same MFMA with the
// dequantised int8 weights rounded to bf16, so every weight of W_hat meets
// its activation as bf16 exactly once.
//
// Split K: when weight blocks x token tiles alone would leave the chip mostly
// idle, the K steps are divided over ksplit blocks per tile (grid z). Splits
// z < ksplit - 1 store their fp32 partial tile as flagged 64-bit slots
// {1, value} (device-coherent stores, no fence) and exit; the last split,
// dispatched after all the others, polls the slots, sums the partials in
// split order (so the result does not depend on timing), clears the slots,
// and runs the epilogue.
#include <algorithm>
#include <type_traits>

#include "bsq_internal.h"

namespace bsq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int BK = 128;    // inputs per K step

// The flagged partial slots sit at a fixed place, the first GEMM_SLOT_BYTES
// of the workspace, whatever the shape: every call leaves them at zero, and
// no other data of any GEMM call is ever written there, so one workspace
// serves calls of different shapes. The K split is capped to fit.
constexpr int64_t GEMM_SLOT_BYTES = int64_t(8) << 20;
// polls of the finishing split for the other splits' slots before it gives
// up and writes NaN (seconds; never expected)
constexpr int GEMM_SPIN_LIMIT = 1 << 22;

struct GemmArgs {
    const void *codes[BSQ_MAX_STAGES];
    const uint16_t *gains[BSQ_MAX_STAGES];
    const uint16_t *tabh[BSQ_MAX_STAGES];  // fp16 decoder tables [2^b][d]
    const int8_t *q8;
    const float *scale;
    const uint16_t *Xt;   // X~ [Mp][Kp]
    const uint16_t *Xp;   // X[:, idx] [Mp][kp32]
    const uint16_t *B;    // LoRA B [d_out][rank]
    const float *T;       // LoRA X A^T [Mp][16]
    int rank;
    int64_t M, d_out, pitch, ksteps, Kp, k, kp32, ldy;
    void *Y;
    int y_bf16;
    int ksplit;        // blocks per tile along K (grid z)
    uint64_t *slots;   // [tiles][ksplit - 1][BM * BN] flagged partials, zero between calls
};

// ---------------------------------------------------------------------------
// Prep: one block per padded token row m < Mp.
// ---------------------------------------------------------------------------
struct PrepArgs {
    const uint16_t *X;
    int64_t ldx, M, d_in, Kp, k, kp32;
    const int32_t *idx;
    const uint16_t *A;  // LoRA A [rank][d_in] or null
    int rank;
    uint16_t *Xt;
    uint16_t *Xp;
    float *T;
};

__global__ __launch_bounds__(256) void gemm_prep(const PrepArgs a)
{
    extern __shared__ uint32_t s_bits[];  // [Kp / 32] protected bitmap
    __shared__ float s_red[BSQ_MAX_LORA_RANK][4];
    const int t = threadIdx.x;
    const int64_t m = blockIdx.x;
    const bool live = m < a.M;
    const int64_t words = a.Kp / 32;
    for (int64_t w = t; w < words; w += 256) s_bits[w] = 0u;
    __syncthreads();
    for (int64_t p = t; p < a.k; p += 256) {
        const int32_t j = a.idx[p];
        if (j >= 0 && j < a.d_in) atomicOr(&s_bits[j >> 5], 1u << (j & 31));
    }
    __syncthreads();
    const uint16_t *xr = a.X + m * a.ldx;
    // X~: 8-input segments; protected inputs, inputs past d_in and rows past
    // M are zero
    for (int64_t sg = t; sg < a.Kp / 8; sg += 256) {
        const int64_t j0 = sg * 8;
        u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
        if (live && j0 < a.d_in) {
            v = *reinterpret_cast<const u32x4_t *>(xr + j0);
            const uint32_t pm = (s_bits[j0 >> 5] >> (j0 & 31)) & 0xffu;
            if (pm) {
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const uint32_t keep = (((pm >> (2 * h)) & 1u) ? 0u : 0xffffu) | (((pm >> (2 * h + 1)) & 1u) ? 0u : 0xffff0000u);
                    v[h] &= keep;
                }
            }
        }
        *reinterpret_cast<u32x4_t *>(a.Xt + m * a.Kp + j0) = v;
    }
    // gathered protected activations, zero past k
    for (int64_t p = t; p < a.kp32; p += 256) {
        uint16_t v = 0;
        if (live && p < a.k) {
            const int32_t j = a.idx[p];
            if (j >= 0 && j < a.d_in) v = xr[j];
        }
        a.Xp[m * a.kp32 + p] = v;
    }
    // T[m][r] = sum_j X[m][j] A[r][j] (fp32), rows past M zero
    if (a.rank > 0) {
        float acc[BSQ_MAX_LORA_RANK];
#pragma unroll
        for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r) acc[r] = 0.0f;
        if (live)
            for (int64_t j = t; j < a.d_in; j += 256) {
                const float x = bf16_to_f32(xr[j]);
#pragma unroll
                for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r)
                    if (r < a.rank) acc[r] = __builtin_fmaf(x, bf16_to_f32(a.A[int64_t(r) * a.d_in + j]), acc[r]);
            }
        const int lane = t & 63, wave = t >> 6;
#pragma unroll
        for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r) {
            float v = acc[r];
            for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
            if (lane == 0) s_red[r][wave] = v;
        }
        __syncthreads();
        if (t < BSQ_MAX_LORA_RANK)
            a.T[m * BSQ_MAX_LORA_RANK + t] = (t < a.rank) ? ((s_red[t][0] + s_red[t][1]) + (s_red[t][2] + s_red[t][3])) : 0.0f;
    }
}

// ---------------------------------------------------------------------------
// Main kernel.
// ---------------------------------------------------------------------------

// Workgroup barrier for LDS traffic only: waits for this wave's LDS (and
// scalar) operations, not for its global loads, which stay in flight across
// the barrier (__syncthreads would drain them with its release fence).
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0), vmcnt and expcnt unconstrained
    asm volatile("s_barrier" ::: "memory");
}

// One K step's code and gain words of a lane, for each of its NT row groups:
// d = 8: chunks 4 g .. 4 g + 3 of the step (one code word, two gain words);
// d = 16: chunks 2 g, 2 g + 1 (one word of two codes, one gain word).
template <int D, int S, int NT>
struct WRegs {
    uint32_t code[NT][S];
    uint32_t gain[NT][S][D == 8 ? 2 : 1];
};

// Number of vector-memory instructions w_load issues (for the wait counts).
template <int D, int S, int NT>
constexpr int w_loads() { return NT * S * 2; }

template <int D, int S, int NT>
__device__ __forceinline__ void w_load(WRegs<D, S, NT> &w, const GemmArgs &a, const int64_t (&ebase)[NT], int64_t ks)
{
    constexpr int CPS = BK / D;
    const int64_t c0 = ks * CPS;
    const int64_t off = ((c0 >> 4) << 10) + (c0 & 15);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int64_t e = ebase[j] + off;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            if constexpr (D == 8) {
                w.code[j][s] = *reinterpret_cast<const uint32_t *>(static_cast<const uint8_t *>(a.codes[s]) + e);
                const uint2 g = *reinterpret_cast<const uint2 *>(a.gains[s] + e);
                w.gain[j][s][0] = g.x;
                w.gain[j][s][1] = g.y;
            } else {
                w.code[j][s] = *reinterpret_cast<const uint32_t *>(static_cast<const uint16_t *>(a.codes[s]) + e);
                w.gain[j][s][0] = *reinterpret_cast<const uint32_t *>(a.gains[s] + e);
            }
        }
    }
}

// B fragments of one row group: bq[q] = the 8 bf16 weights of inputs
// 32 g + 8 q .. + 8 of the step (d = 8: chunk 4 g + q; d = 16: half q % 2 of
// chunk 2 g + q / 2), each sum_s gain_s * D_s(code_s)[j] as an fp32 fmaf
// chain over fp16 gains and fp16 table values (v_fma_mix_f32), rounded to
// bf16. d = 8 reads the tables from LDS, d = 16 from global memory.
template <int D, int S, int NT>
__device__ __forceinline__ void w_decode(const WRegs<D, S, NT> &w, int j, const GemmArgs &a, const uint16_t *s_tab,
                                         u32x4_t (&bq)[4])
{
    typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
    constexpr int CPL = (D == 8) ? 4 : 2;  // chunks per lane
#pragma unroll
    for (int u = 0; u < CPL; ++u) {
        float v[D];
#pragma unroll
        for (int e = 0; e < D; ++e) v[e] = 0.0f;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const uint32_t code = (D == 8) ? ((w.code[j][s] >> (8 * u)) & 0xffu) : ((w.code[j][s] >> (16 * u)) & 0xffffu);
            const uint32_t gw = (D == 8) ? w.gain[j][s][u >> 1] : w.gain[j][s][0];
            const float g = f16_bits_to_f32(uint16_t((u & 1) ? (gw >> 16) : (gw & 0xffffu)));
            const uint16_t *y = (D == 8) ? (s_tab + (s * 256 + code) * 8) : (a.tabh[s] + size_t(code) * D);
#pragma unroll
            for (int q = 0; q < D / 8; ++q) {
                const f16x8_t yy = *reinterpret_cast<const f16x8_t *>(y + 8 * q);
#pragma unroll
                for (int e = 0; e < 8; ++e) v[8 * q + e] = __builtin_fmaf(g, float(yy[e]), v[8 * q + e]);
            }
        }
#pragma unroll
        for (int h = 0; h < D / 8; ++h)
            bq[(D == 8) ? u : 2 * u + h] = u32x4_t{pack_bf16x2(v[8 * h + 0], v[8 * h + 1]), pack_bf16x2(v[8 * h + 2], v[8 * h + 3]),
                                                   pack_bf16x2(v[8 * h + 4], v[8 * h + 5]), pack_bf16x2(v[8 * h + 6], v[8 * h + 7])};
    }
}

// One block: BN = 64 NT rows x BM = 16 MT tokens x the K steps [kb, ke) of
// split z. Wave w owns rows 16 (NT w + j) + lane % 16 of the block, j < NT,
// and all BM tokens: acc[i][j] element r is token 16 i + 4 (lane / 16) + r.
template <int D, int S, int MT, int NT>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmArgs a)
{
    constexpr int BM = MT * 16, BN = 64 * NT;
    constexpr int XSLOT = BM * BK;   // bf16 elements per X~ slot
    constexpr int NXL = BM / 16;     // X~ loads (16 B) per lane per step
    constexpr int NW = w_loads<D, S, NT>();
    static_assert(NW <= 63, "wait count fits vmcnt");
    // LDS: two X~ slots [BM][128] bf16 (the 16-byte segment s of row r
    // stored at position s ^ (r % 16): conflict-free fragment reads), and the
    // fp32 tables (D == 8)
    __shared__ __attribute__((aligned(16))) uint16_t s_x[2][XSLOT];
    __shared__ __attribute__((aligned(16))) uint16_t s_tab[(D == 8) ? S * 2048 : 8];

    const int t = threadIdx.x, lane = t & 63, g = lane >> 4;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int64_t n0 = int64_t(blockIdx.x) * BN;          // first row of the block
    const int64_t m0 = int64_t(blockIdx.y) * BM;          // first token of the block
    const int z = blockIdx.z;
    const int64_t kb = a.ksteps * z / a.ksplit, ke = a.ksteps * (z + 1) / a.ksplit;
    const int64_t nb = a.pitch / 16;
    int64_t ebase[NT];  // tile element of the lane's row, chunk group g, step 0
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int64_t row = n0 + 16 * (NT * wave + j) + (lane & 15);
        ebase[j] = (((row >> 6) * nb) << 10) + ((row & 63) << 4) + (BK / D / 4) * g;
    }

    // fp16 tables (D == 8): S x 2048 values, one 16-byte piece per thread
    // per stage, all loads issued before the first store
    if constexpr (D == 8) {
        u32x4_t tv[S];
#pragma unroll
        for (int s = 0; s < S; ++s) tv[s] = reinterpret_cast<const u32x4_t *>(a.tabh[s])[t];
#pragma unroll
        for (int s = 0; s < S; ++s) reinterpret_cast<u32x4_t *>(s_tab + s * 2048)[t] = tv[s];
    }

    f32x4_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // X~ tile of step ks through registers: pass n of thread t carries the
    // 16-byte segment e = 256 n + t, row e / 16, segment e % 16
    auto x_load = [&](u32x4_t (&xr)[NXL], int64_t ks) {
#pragma unroll
        for (int n = 0; n < NXL; ++n) {
            const int e = 256 * n + t;
            xr[n] = *reinterpret_cast<const u32x4_t *>(a.Xt + (m0 + (e >> 4)) * a.Kp + ks * BK + 8 * (e & 15));
        }
    };
    auto x_store = [&](const u32x4_t (&xr)[NXL], uint16_t *slot) {
#pragma unroll
        for (int n = 0; n < NXL; ++n) {
            const int e = 256 * n + t, r = e >> 4;
            *reinterpret_cast<u32x4_t *>(slot + r * BK + 8 * ((e & 15) ^ (r & 15))) = xr[n];
        }
    };

    // One K step ks at parity P: wait until only the code and gain loads of
    // step ks + 1 may be in flight (issue order per step: X~ of step ks + 2,
    // then code and gain words of step ks + 2), barrier, store X~ of step
    // ks + 1 to the other slot (read last in step ks - 1, before this
    // barrier), issue the loads of step ks + 2 (clamped to the last step: a
    // harmless reload), decode this step's weights, MFMAs on this step's slot.
    WRegs<D, S, NT> w[2];
    u32x4_t xr[2][NXL];
    auto step = [&](auto pc, int64_t ks) {
        constexpr int P = decltype(pc)::value;
        __builtin_amdgcn_s_waitcnt((NW & 15) | ((NW >> 4) << 14) | (7 << 4) | (15 << 8));
        lds_barrier();
        x_store(xr[P ^ 1], s_x[P ^ 1]);
        const int64_t kn = (ks + 2 < ke) ? ks + 2 : ke - 1;
        x_load(xr[P], kn);
        // keep the issue order (X~ loads, decode, code and gain loads): the
        // wait at the top of the next step relies on it
        __builtin_amdgcn_sched_barrier(0);
        u32x4_t bq[NT][4];
#pragma unroll
        for (int j = 0; j < NT; ++j) w_decode<D, S, NT>(w[P], j, a, s_tab, bq[j]);
        __builtin_amdgcn_sched_barrier(0);
        w_load<D, S, NT>(w[P], a, ebase, kn);
        __builtin_amdgcn_sched_barrier(0);
        const uint16_t *xs = s_x[P];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const int rr = 16 * i + (lane & 15);
                const u32x4_t av = *reinterpret_cast<const u32x4_t *>(xs + rr * BK + 8 * ((4 * g + q) ^ (lane & 15)));
                const bf16x8_t aop = __builtin_bit_cast(bf16x8_t, av);
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(aop, __builtin_bit_cast(bf16x8_t, bq[j][q]), acc[i][j], 0, 0, 0);
            }
        }
    };
    // prologue: X~ of step kb in its slot, step kb + 1 in registers, code and
    // gain words of kb and kb + 1 in flight (kb + 1 clamped)
    const int64_t k1 = (kb + 1 < ke) ? kb + 1 : ke - 1;
    x_load(xr[0], kb);
    w_load<D, S, NT>(w[0], a, ebase, kb);
    x_load(xr[1], k1);
    w_load<D, S, NT>(w[1], a, ebase, k1);
    x_store(xr[0], s_x[0]);
    for (int64_t ks = kb; ks < ke; ks += 2) {
        step(std::integral_constant<int, 0>(), ks);
        if (ks + 1 < ke) step(std::integral_constant<int, 1>(), ks + 1);
    }
    __builtin_amdgcn_s_waitcnt(0);  // loads past the last step land before the block ends

    // protected term (split 0 only): X[:, idx] (bf16) times bf16(q8 s), the
    // weights of lane row 16 (NT w + j) + lane % 16 at positions 32 qq + 8 g + e
    if (z == 0 && a.k > 0) {
        const int64_t kp = q8_pitch(a.k);
        for (int64_t qq = 0; qq < a.kp32 / 32; ++qq) {
            const int64_t p0 = 32 * qq + 8 * g;
            u32x4_t bp[NT];
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const int64_t row = n0 + 16 * (NT * wave + j) + (lane & 15);
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int64_t p = p0 + e;
                    v[e] = (row < a.d_out && p < a.k) ? float(a.q8[row * kp + p]) * a.scale[p] : 0.0f;
                }
                bp[j] = u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
            }
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                const u32x4_t av = *reinterpret_cast<const u32x4_t *>(a.Xp + (m0 + 16 * i + (lane & 15)) * a.kp32 + p0);
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av),
                                                                         __builtin_bit_cast(bf16x8_t, bp[j]), acc[i][j], 0, 0, 0);
            }
        }
    }

    bool timed_out = false;
    if (a.ksplit > 1) {
        // partial tile in MFMA fragment order: slot ((wave MT + i) NT + j) 256
        // + 64 r + lane of the split's [BM * BN] range
        const int64_t tile = int64_t(blockIdx.y) * gridDim.x + blockIdx.x;
        uint64_t *tp = a.slots + tile * int64_t(a.ksplit - 1) * (BM * BN) + lane;
        auto slot = [&](int zz, int i, int j, int r) { return tp + int64_t(zz) * (BM * BN) + ((wave * MT + i) * NT + j) * 256 + 64 * r; };
        if (z < a.ksplit - 1) {
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < NT; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        __hip_atomic_store(slot(z, i, j, r), (uint64_t(1) << 32) | __float_as_uint(acc[i][j][r]),
                                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return;
        }
        // the finishing split: partials of splits 0 .. ksplit - 2 in order,
        // then its own
        f32x4_t sum[MT][NT];
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) sum[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
        for (int zz = 0; zz < a.ksplit - 1; ++zz) {
            uint64_t pw[MT][NT][4];
            for (int spin = 0;; ++spin) {
                bool ready = true;
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            pw[i][j][r] = __hip_atomic_load(slot(zz, i, j, r), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            ready &= (pw[i][j][r] >> 32) != 0;
                        }
                if (__all(ready)) break;
                if (spin == GEMM_SPIN_LIMIT) {  // never expected: report NaN rather than hang
                    timed_out = true;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < NT; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        sum[i][j][r] += __uint_as_float(uint32_t(pw[i][j][r]));
                        __hip_atomic_store(slot(zz, i, j, r), uint64_t(0), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
        }
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) acc[i][j] = sum[i][j] + acc[i][j];
    }

    // epilogue: LoRA, then Y
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int64_t n = n0 + 16 * (NT * wave + j) + (lane & 15);
        if (n >= a.d_out) continue;
        float bl[BSQ_MAX_LORA_RANK];
#pragma unroll
        for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) bl[q] = (q < a.rank) ? bf16_to_f32(a.B[n * a.rank + q]) : 0.0f;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int64_t m = m0 + 16 * i + 4 * g + r;
                if (m >= a.M) continue;
                float v = timed_out ? __builtin_nanf("") : acc[i][j][r];
                if (a.rank > 0) {
                    const float *Tm = a.T + m * BSQ_MAX_LORA_RANK;
#pragma unroll
                    for (int q = 0; q < BSQ_MAX_LORA_RANK; ++q) v = __builtin_fmaf(bl[q], Tm[q], v);
                }
                if (a.y_bf16) static_cast<uint16_t *>(a.Y)[m * a.ldy + n] = f32_to_bf16(v);
                else static_cast<float *>(a.Y)[m * a.ldy + n] = v;
            }
        }
    }
}

// Launch shape: token tile and rows per block by M, then the K split, then
// the workspace layout.
struct GemmPlan {
    int mt, nt;  // token groups and 64-row groups per block
    int64_t bm, bn, mtiles, nblk, ksteps, ksplit, Mp, Kp, kp32;
    size_t t_off, xt_off, xp_off, total;
};

GemmPlan gemm_plan(int64_t d_out, int64_t d_in, int64_t M, int64_t k)
{
    GemmPlan p{};
    int occ;  // blocks per CU the variant reaches (LDS)
    if (M <= 16) p.mt = 1, p.nt = 1, occ = 4;
    else if (M <= 64) p.mt = 4, p.nt = 2, occ = 2;
    else p.mt = 8, p.nt = 2, occ = 1;
    p.bm = 16 * p.mt;
    p.bn = 64 * p.nt;
    p.mtiles = (M + p.bm - 1) / p.bm;
    p.nblk = (d_out + p.bn - 1) / p.bn;
    p.ksteps = (d_in + BK - 1) / BK;
    p.Mp = std::max<int64_t>(p.mtiles, 1) * p.bm;
    p.Kp = p.ksteps * BK;
    p.kp32 = (k + 31) & ~int64_t(31);
    const int64_t tiles = p.nblk * p.mtiles;
    // about two rounds of blocks over 256 CUs, at least 4 K steps per block,
    // the flagged partials within GEMM_SLOT_BYTES
    int64_t ks = (2 * 256 * occ + tiles - 1) / (tiles > 0 ? tiles : 1);
    ks = std::min<int64_t>(ks, p.ksteps / 4);
    ks = std::min<int64_t>(ks, 1 + GEMM_SLOT_BYTES / std::max<int64_t>(1, tiles * p.bm * p.bn * 8));
    ks = std::min<int64_t>(ks, 64);
    p.ksplit = std::max<int64_t>(ks, 1);
    p.t_off = size_t(GEMM_SLOT_BYTES);
    p.xt_off = p.t_off + align256(size_t(p.Mp) * BSQ_MAX_LORA_RANK * 4);
    p.xp_off = p.xt_off + align256(size_t(p.Mp) * size_t(p.Kp) * 2);
    p.total = p.xp_off + align256(size_t(p.Mp) * size_t(std::max<int64_t>(p.kp32, 32)) * 2);
    return p;
}

template <int D, int S, int MT, int NT>
hipError_t launch_main(const GemmArgs &a, const GemmPlan &p, hipStream_t st)
{
    const dim3 grid = dim3(unsigned(p.nblk), unsigned(p.mtiles), unsigned(p.ksplit));
    hipLaunchKernelGGL((gemm_kernel<D, S, MT, NT>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int D, int S>
hipError_t launch_gemm_t(const GemmArgs &a, const GemmPlan &p, hipStream_t st)
{
    if (p.mt == 1) return launch_main<D, S, 1, 1>(a, p, st);
    if (p.mt == 4) return launch_main<D, S, 4, 2>(a, p, st);
    return launch_main<D, S, 8, 2>(a, p, st);
}

}  // namespace

size_t gemm_ws_bytes(const bsq_config &cfg, int64_t d_out, int64_t d_in, int64_t M)
{
    const int64_t k = cfg.protect_num ? (d_in * cfg.protect_num + cfg.protect_den - 1) / cfg.protect_den : 0;
    return gemm_plan(d_out, d_in, M, k).total;
}

hipError_t launch_gemm(const bsq_config &cfg, const void *codec, const bsq_layer &L, const bsq_lora *lora,
                       const void *X, int64_t M, int64_t ldx, void *Y, int y_dtype, int64_t ldy, void *ws,
                       hipStream_t st)
{
    if (M == 0 || L.d_out == 0) return hipSuccess;
    const GemmPlan p = gemm_plan(L.d_out, L.d_in, M, L.k);
    char *wb = static_cast<char *>(ws);
    GemmArgs a{};
    const char *cb = static_cast<const char *>(codec);
    for (int s = 0; s < cfg.stages; ++s) {
        a.codes[s] = L.codes[s];
        a.gains[s] = L.gains[s];
        a.tabh[s] = reinterpret_cast<const uint16_t *>(cb + codec_tabh_offset(cfg, s));
    }
    a.q8 = L.prot_q8;
    a.scale = L.prot_scale;
    a.Xt = reinterpret_cast<const uint16_t *>(wb + p.xt_off);
    a.Xp = reinterpret_cast<const uint16_t *>(wb + p.xp_off);
    a.T = reinterpret_cast<const float *>(wb + p.t_off);
    a.M = M;
    a.d_out = L.d_out;
    a.pitch = L.pitch;
    a.ksteps = p.ksteps;
    a.Kp = p.Kp;
    a.k = L.k;
    a.kp32 = p.kp32;
    a.ldy = ldy;
    a.Y = Y;
    a.y_bf16 = (y_dtype == BSQ_BF16);
    a.rank = 0;
    a.ksplit = int(p.ksplit);
    a.slots = static_cast<uint64_t *>(ws);

    PrepArgs pa{};
    pa.X = static_cast<const uint16_t *>(X);
    pa.ldx = ldx;
    pa.M = M;
    pa.d_in = L.d_in;
    pa.Kp = p.Kp;
    pa.k = L.k;
    pa.kp32 = p.kp32;
    pa.idx = L.prot_idx;
    pa.Xt = reinterpret_cast<uint16_t *>(wb + p.xt_off);
    pa.Xp = reinterpret_cast<uint16_t *>(wb + p.xp_off);
    pa.T = reinterpret_cast<float *>(wb + p.t_off);
    if (lora && lora->rank > 0) {
        a.rank = lora->rank;
        a.B = lora->B;
        pa.A = lora->A;
        pa.rank = lora->rank;
    }
    hipLaunchKernelGGL(gemm_prep, dim3(unsigned(p.Mp)), dim3(256), size_t(p.Kp / 32) * 4, st, pa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    const int S = cfg.stages;
    if (cfg.d == 8) {
        switch (S) {
        case 1: return launch_gemm_t<8, 1>(a, p, st);
        case 2: return launch_gemm_t<8, 2>(a, p, st);
        case 3: return launch_gemm_t<8, 3>(a, p, st);
        default: return launch_gemm_t<8, 4>(a, p, st);
        }
    }
    switch (S) {
    case 1: return launch_gemm_t<16, 1>(a, p, st);
    case 2: return launch_gemm_t<16, 2>(a, p, st);
    case 3: return launch_gemm_t<16, 3>(a, p, st);
    default: return launch_gemm_t<16, 4>(a, p, st);
    }
}

}  // namespace bsq
