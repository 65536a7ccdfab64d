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
// fragment q cover inputs 32 g + 8 q .. + 8 of the step. The X~ tile and the
// code and gain words of a K step reach LDS by DMA (global_load_lds) into
// rings of NS slots, issued NS - 1 steps ahead; one barrier per step. The
// protected term X[:, idx] (q8 s)^T and LoRA are added in the epilogue, both
// through the same MFMA: the dequantised int8 weights rounded to bf16 (so
// every weight of W_hat meets its activation as bf16 exactly once), and T
// split exactly into three bf16 parts against bf16 B.
//
// Split K: when weight blocks x token tiles alone would leave the chip mostly
// idle, the K steps are divided over ksplit blocks per tile (grid z). Every
// split stores its fp32 partial tile to a scratch area of the workspace, and
// a second kernel sums the partials in split order (so the result does not
// depend on timing) and stores Y. (A finishing block that gathered the other
// splits' partials itself read them at the rate one compute unit reaches on
// device-coherent loads, 20-30 GB/s, which made a 1024-row projection at 256
// tokens take 55 us.)
#include <algorithm>
#include <type_traits>

#include "bsq_internal.h"

namespace bsq {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int BK = 128;    // inputs per K step

// The workspace starts with a 256-byte header that the product leaves
// untouched (no block of it waits for another, so there is no poison word
// or flagged slot to keep); the scratch of a call follows: T = X A^T, X~, the
// gathered protected activations and the split-K partials.
constexpr int64_t GEMM_HDR = 256;

// Eight stored protected bytes (two words, byte e of the pair at bits
// 8 (e % 4) of word e / 4) times their scales, in format FMT; the run-time
// format is dispatched once per eight bytes (a uniform branch).
template <int FMT>
__device__ __forceinline__ void payload8_t(uint2 qv, const float *sc, float (&v)[8])
{
    v[0] = payload_byte<FMT, 0>(qv.x) * sc[0];
    v[1] = payload_byte<FMT, 1>(qv.x) * sc[1];
    v[2] = payload_byte<FMT, 2>(qv.x) * sc[2];
    v[3] = payload_byte<FMT, 3>(qv.x) * sc[3];
    v[4] = payload_byte<FMT, 0>(qv.y) * sc[4];
    v[5] = payload_byte<FMT, 1>(qv.y) * sc[5];
    v[6] = payload_byte<FMT, 2>(qv.y) * sc[6];
    v[7] = payload_byte<FMT, 3>(qv.y) * sc[7];
}

__device__ __forceinline__ void payload8(uint2 qv, const float *sc, float (&v)[8], int fmt)
{
    if (fmt == BSQ_PROT_E4M3) payload8_t<BSQ_PROT_E4M3>(qv, sc, v);
    else if (fmt == BSQ_PROT_E5M2) payload8_t<BSQ_PROT_E5M2>(qv, sc, v);
    else payload8_t<BSQ_PROT_INT8>(qv, sc, v);
}

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
    int y_vec;         // Y 16-byte aligned with 16-byte row pitch: vector stores
    int ksplit;        // blocks per tile along K (grid z)
    float *part;       // split-K partials [ksplit][Mp][np] (ksplit > 1)
    int64_t np;        // row pitch of the partials (d_out padded to whole blocks)
    int pfmt;          // bsq_prot_format of q8
};

// ---------------------------------------------------------------------------
// Prep: one workgroup per (padded token row m < Mp, block of PREP_COLS X~
// columns); the first column block of a row also writes its protected
// activations and T.
// ---------------------------------------------------------------------------
constexpr int PREP_COLS = 2048;  // X~ columns per prep workgroup (256 threads x 8)
struct PrepArgs {
    const uint16_t *X;
    int64_t ldx, M, d_in, Kp, k, kp32;
    const int32_t *idx;
    const uint32_t *bits;  // protected-column bitmap of the layer (k > 0)
    const uint16_t *A;  // LoRA A [rank][d_in] or null
    int rank;
    uint16_t *Xt;
    uint16_t *Xp;
    float *T;
};

__global__ __launch_bounds__(256) void gemm_prep(const PrepArgs a)
{
    // workgroup (m, y): token row m < Mp; y < ncb: X~ columns [2048 y, 2048 y
    // + 2048); y == ncb: the gathered protected activations (and the zero
    // LoRA entries past the rank); y = ncb + 1 + r: T[m][r] for rank index r
    __shared__ float s_red[4];
    const int t = threadIdx.x;
    const int64_t m = blockIdx.x;
    const int64_t ncb = (a.Kp + PREP_COLS - 1) / PREP_COLS;
    const int64_t y = blockIdx.y;
    const bool live = m < a.M;
    const uint16_t *xr = a.X + m * a.ldx;
    if (y < ncb) {
        // X~: one 8-input segment per thread; protected inputs (the layer's
        // bitmap, read with the segment), inputs past d_in and rows past M
        // are zero
        const int64_t j0 = y * PREP_COLS + 8 * t;
        if (j0 < a.Kp) {
            u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
            if (live && j0 < a.d_in) {
                v = *reinterpret_cast<const u32x4_t *>(xr + j0);
                const uint32_t pm = (a.k > 0 && a.bits) ? (a.bits[j0 >> 5] >> (j0 & 31)) & 0xffu : 0u;
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const uint32_t keep = (((pm >> (2 * h)) & 1u) ? 0u : 0xffffu) | (((pm >> (2 * h + 1)) & 1u) ? 0u : 0xffff0000u);
                    v[h] &= keep;
                }
            }
            *reinterpret_cast<u32x4_t *>(a.Xt + m * a.Kp + j0) = v;
        }
        return;
    }
    if (y == ncb) {
        // gathered protected activations, zero past k
        for (int64_t p = t; p < a.kp32; p += 256) {
            uint16_t v = 0;
            if (live && p < a.k) {
                const int32_t j = a.idx[p];
                if (j >= 0 && j < a.d_in) v = xr[j];
            }
            a.Xp[m * a.kp32 + p] = v;
        }
        // LoRA entries past the rank (all of them without an adapter) are zero
        if (t >= a.rank && t < BSQ_MAX_LORA_RANK) a.T[m * BSQ_MAX_LORA_RANK + t] = 0.0f;
        return;
    }
    // T[m][r] = sum_j X[m][j] A[r][j] (fp32, exact bf16 products), rows past M
    // zero: eight inputs per 16-byte load where the row of A is 16-byte
    // aligned, four loads per thread in flight, element by element elsewhere
    const int r = int(y - ncb - 1);
    const uint16_t *ar = a.A + int64_t(r) * a.d_in;
    float acc = 0.0f;
    if (live) {
        const bool vec = (reinterpret_cast<uintptr_t>(ar) & 15) == 0;
        const int64_t n8 = vec ? a.d_in / 8 : 0;
        for (int64_t p0 = t; p0 < n8; p0 += 4 * 256) {
            u32x4_t av[4], xv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t p = (p0 + u * 256 < n8) ? p0 + u * 256 : n8 - 1;
                av[u] = reinterpret_cast<const u32x4_t *>(ar)[p];
                xv[u] = reinterpret_cast<const u32x4_t *>(xr)[p];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                if (p0 + u * 256 >= n8) break;
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    acc = __builtin_fmaf(__uint_as_float(av[u][h] << 16), __uint_as_float(xv[u][h] << 16), acc);
                    acc = __builtin_fmaf(__uint_as_float(av[u][h] & 0xffff0000u), __uint_as_float(xv[u][h] & 0xffff0000u),
                                         acc);
                }
            }
        }
        for (int64_t j = n8 * 8 + t; j < a.d_in; j += 256) acc = __builtin_fmaf(bf16_to_f32(xr[j]), bf16_to_f32(ar[j]), acc);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if ((t & 63) == 0) s_red[t >> 6] = acc;
    __syncthreads();
    if (t == 0) a.T[m * BSQ_MAX_LORA_RANK + r] = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
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

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm()
{
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// LDS of one workgroup (gfx950: 160 KiB per compute unit).
constexpr int GEMM_LDS_BYTES = 160 * 1024;

// Workgroups per compute unit of the main kernel. The 16-token, 64-row block
// (56-74 VGPRs) runs three where three fit in LDS (4 ring slots of X~ and
// weight words each, plus one table copy at d = 8, where 1 or 2 stages fit;
// the d = 16 tables stay in global memory): its steps are short, and three
// blocks' waits (the DMAs, and at d = 16 the table gathers) overlap. The
// 64-token block (100-122 VGPRs) runs two where two fit with at least two
// ring slots each (up to four). Every other shape runs one, with as many
// ring slots as fit. The plan sizes its K splits by the same count.
constexpr int gemm_wg_per_cu(int d, int s, int mt, int nt)
{
    if (mt == 4)
        return (2 * (2 * (16 * mt * 256 + nt * s * (d == 8 ? 192 : 128) * 16) + (d == 8 ? s * 4096 : 0)) <= GEMM_LDS_BYTES)
                   ? 2 : 1;
    if (mt != 1 || nt != 1) return 1;
    if (d == 16) return 3;
    return (d == 8 && 3 * (4 * (16 * mt * 256 + nt * s * 192 * 16) + s * 4096) <= GEMM_LDS_BYTES) ? 3 : 1;
}

// Shape of the main kernel. A workgroup of 8 waves owns BN = 64 NT weight
// rows and BM = 16 MT tokens. Wave w owns the row set rs = w % 4 (NT groups of
// 16 rows: block rows 16 (NT rs + j) + lane % 16) and the half kh = w / 4 of
// every K step (MFMA k-slices 2 kh and 2 kh + 1); the two halves of a row
// set add their tiles at the end. Per K step, the X~ tile and the code and
// gain words of the block's NT 64-row plane tiles reach LDS by DMA
// (global_load_lds_dwordx4, 64 16-byte units per wave instruction) into a
// ring of NS slots, NS - 1 steps ahead.
template <int D, int S, int MT, int NT>
struct GemmShape {
    static constexpr int BM = 16 * MT, BN = 64 * NT;
    // 16-byte units of one (64-row tile, stage) per step: d = 8, the tile's
    // 1 KiB of codes and 2 KiB of gains; d = 16, half a tile (the step's 8
    // chunks): 16 bytes of codes and 16 of gains per row
    static constexpr int WU = (D == 8) ? 192 : 128;
    static constexpr int XSLOT = BM * 256;            // bytes: [BM][128] bf16
    static constexpr int WSLOT = NT * S * WU * 16;    // bytes: [NT][S][codes | gains]
    static constexpr int WG_PER_CU = gemm_wg_per_cu(D, S, MT, NT);
    // fp16 decoder tables (d = 8) [S][256 codes][TC copies][8]: lane l reads
    // copy l % TC, which spreads the random lookups of a wave over the LDS
    // banks; 8 copies where three ring slots still fit, else one
    static constexpr int TC = (D == 8 && WG_PER_CU == 1 && (GEMM_LDS_BYTES - S * 4096 * 8) / (XSLOT + WSLOT) >= 3) ? 8 : 1;
    static constexpr int TAB = (D == 8) ? S * 4096 * TC : 0;
    static constexpr int NS_FIT = (GEMM_LDS_BYTES / WG_PER_CU - TAB) / (XSLOT + WSLOT);
    static constexpr int NS = (WG_PER_CU > 1) ? (NS_FIT < 4 ? NS_FIT : 4) : NS_FIT < 8 ? NS_FIT : 8;
    static constexpr int NXI = BM / 4;              // X~ DMA wave instructions per step
    static constexpr int NWI = NT * S * WU / 64;    // weight DMA wave instructions per step
    static constexpr int NI = NXI + NWI;            // wave w issues instructions w, w + 8, ... < NI
    static constexpr int PMAX = (NI + 7) / 8, PMIN = NI / 8;  // DMA instructions per wave and step
    static constexpr size_t LDS = size_t(NS) * (XSLOT + WSLOT) + TAB;
    static_assert(NS >= 2, "two pipeline stages fit in LDS");
    static_assert(LDS * WG_PER_CU <= size_t(GEMM_LDS_BYTES), "the workgroups of a compute unit fit in its LDS");
    static_assert(MT * NT * 4096 <= NS * XSLOT, "the exchange of the two K halves fits in the X~ ring");
    static_assert((NS - 1) * PMAX <= 63, "wait count fits vmcnt");
    static_assert(WU % 64 == 0, "a DMA instruction stays within one (tile, stage)");
};

// One block: BN rows x BM tokens x the K steps [kb, ke) of split z.
// acc[i][j] element r is token 16 i + 4 (lane / 16) + r of row group j.
//
// K step ks (slot ks % NS of both rings): wait until only the DMAs of the
// next NS - 2 steps may be in flight, barrier (every wave's DMAs of step ks
// have landed, and every wave is done with step ks - 1), DMA step
// ks + NS - 1 into the slot step ks - 1 used (clamped to the last step: a
// harmless reload into a free slot), decode this wave's B fragments from the
// slot's code and gain words and the LDS tables, MFMAs against the X~ slot.
// The inputs of a step are permuted identically on both operands so that a
// lane's fragment is a whole chunk (d = 8) or half a chunk (d = 16): MFMA
// input group g = lane / 16 of k-slice q covers inputs 32 g + 8 q .. + 8.
template <int D, int S, int MT, int NT>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(GemmShape<D, S, MT, NT>::WG_PER_CU * 2)))
void gemm_kernel(const GemmArgs a)
{
    using G = GemmShape<D, S, MT, NT>;
    typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
    extern __shared__ __attribute__((aligned(16))) uint4 s_mem4[];
    uint8_t *s_mem = reinterpret_cast<uint8_t *>(s_mem4);
    uint8_t *s_xr = s_mem;                          // X~ ring (MFMA fragment order)
    uint8_t *s_wr = s_mem + G::NS * G::XSLOT;       // weight ring
    uint4 *s_tab4 = reinterpret_cast<uint4 *>(s_wr + G::NS * G::WSLOT);  // d = 8 tables
    const uint16_t *s_tab = reinterpret_cast<const uint16_t *>(s_tab4);

    const int t = threadIdx.x, lane = t & 63, g = lane >> 4, r16 = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int rs = wave & 3, kh = wave >> 2;
    // Tile of the block. The workgroups of a launch go to the 8 XCDs in turn
    // (linear id mod 8), each XCD with its own L2. With K split and token
    // tiles of 64 or more, consecutive tiles in (token tile, row block,
    // split) order are given to one XCD, so that an XCD reads only its splits'
    // share of X~ and keeps both token tiles of a row block (which share its
    // weights); a bijection whenever the block count is a multiple of 8.
    int bx = blockIdx.x, by = blockIdx.y, bz = blockIdx.z;
    if (MT >= 4 && a.ksplit > 1) {
        const int nx = gridDim.x, ny = gridDim.y, total = nx * ny * int(gridDim.z);
        if ((total & 7) == 0) {
            const int lin = bx + nx * (by + ny * bz);
            const int lg = (lin & 7) * (total >> 3) + (lin >> 3);
            by = lg % ny;
            bx = (lg / ny) % nx;
            bz = lg / (ny * nx);
        }
    }
    const int64_t n0 = int64_t(bx) * G::BN;  // first row of the block
    const int64_t m0 = int64_t(by) * G::BM;  // first token of the block
    const int z = bz;
    const int64_t kb = a.ksteps * z / a.ksplit, ke = a.ksteps * (z + 1) / a.ksplit;
    const int64_t nb = a.pitch / 16;                 // 16-chunk blocks per row
    const int64_t rbmax = (a.d_out + 63) / 64 - 1;   // last 64-row tile of the planes

    // DMA instructions of this wave, r-th: joint instruction v = wave + 8 r
    // of the step (v < NXI: 64 units of X~, unit u = row u / 16, LDS segment
    // u % 16; else 64 units of the code and gain words of (64-row tile jt,
    // stage s), tiles past the planes clamped to the last one, whose rows are
    // never stored). Source of step ks = base + (ks / 2) A + (ks % 2) B bytes;
    // destination = ring + slot * slot bytes + offset.
    const uint8_t *dsrc[G::PMAX];
    int64_t dA[G::PMAX], dB[G::PMAX];
    int doff[G::PMAX], dslot[G::PMAX];
    bool dx[G::PMAX];
#pragma unroll
    for (int r = 0; r < G::PMAX; ++r) {
        const int v0 = wave + 8 * r;
        const int v = (v0 < G::NI) ? v0 : G::NI - 1;  // (r-th instruction absent when v0 >= NI)
        if (v < G::NXI) {
            // X~ slot in MFMA fragment order: unit (q MT + i) 64 + l holds the
            // 8 inputs 32 (l / 16) + 8 q of token 16 i + l % 16 (k-slice q)
            const int q = v / MT, i = v - q * MT;
            dsrc[r] = reinterpret_cast<const uint8_t *>(a.Xt + (m0 + 16 * i + r16) * a.Kp + 32 * g + 8 * q);
            dA[r] = 2 * 2 * BK;
            dB[r] = 2 * BK;
            dx[r] = true;
            doff[r] = 1024 * v;
            dslot[r] = G::XSLOT;
        } else {
            const int vw = v - G::NXI;
            const int pair = (64 * vw) / G::WU;        // jt * S + s (uniform over the wave)
            const int w0 = 64 * vw - pair * G::WU;     // first unit within the (tile, stage)
            const int jt = pair / S, st = pair - jt * S;
            const int64_t rb = ((n0 >> 6) + jt < rbmax) ? (n0 >> 6) + jt : rbmax;
            const int w = w0 + lane;
            const int64_t tb = (rb * nb) << 10;        // element of the row block's first tile
            if constexpr (D == 8) {
                dsrc[r] = (w0 < 64) ? static_cast<const uint8_t *>(a.codes[st]) + tb + 16 * w
                                    : reinterpret_cast<const uint8_t *>(a.gains[st] + tb) + 16 * (w - 64);
                dA[r] = (w0 < 64) ? 2048 : 4096;
                dB[r] = (w0 < 64) ? 1024 : 2048;
            } else {
                dsrc[r] = (w0 < 64) ? reinterpret_cast<const uint8_t *>(static_cast<const uint16_t *>(a.codes[st]) + tb) + 32 * (w & 63)
                                    : reinterpret_cast<const uint8_t *>(a.gains[st] + tb) + 32 * (w & 63);
                dA[r] = 2048;
                dB[r] = 16;
            }
            dx[r] = false;
            doff[r] = 1024 * vw;
            dslot[r] = G::WSLOT;
        }
    }
    const int pw = (wave < G::NI % 8) ? G::PMAX : G::PMIN;  // this wave's DMA instructions per step
    // issue group: X~ of step kx into X~ slot slx and the weights of step kw
    // into weight slot slw (w_only: the weights alone)
    auto dma_group = [&](int64_t kx, int slx, int64_t kw, int slw, bool w_only) {
#pragma unroll
        for (int r = 0; r < G::PMAX; ++r) {
            if (r >= G::PMIN && wave + 8 * r >= G::NI) continue;
            if (w_only && dx[r]) continue;
            const int64_t k = dx[r] ? kx : kw;
            const uint4 *src = reinterpret_cast<const uint4 *>(dsrc[r] + (k >> 1) * dA[r] + (k & 1) * dB[r]);
            uint8_t *dst = dx[r] ? s_xr + slx * G::XSLOT + doff[r] : s_wr + slw * G::WSLOT + doff[r];
            __builtin_amdgcn_global_load_lds(src, reinterpret_cast<uint4 *>(dst), 16, 0, 0);
        }
    };
    auto clampk = [&](int64_t k) { return (k < ke) ? k : ke - 1; };

    // Software pipeline over the K steps. Group c (c >= 0) carries the X~ of
    // step kb + c (X~ slot c % NS) and the weights of step kb + c + 1 (weight
    // slot (c + 1) % NS); group -1 the weights of step kb. Iteration c runs
    // the MFMAs of step kb + c with B fragments decoded in iteration c - 1
    // while it decodes step kb + c + 1, so the matrix cores and the decode
    // arithmetic overlap. Steps past ke - 1 are clamped (harmless reloads
    // into slots no later iteration reads before they are refilled).
    if constexpr (D == 8) {
        // decoder tables: wave instruction v fills LDS units 64 v .. + 63, unit
        // (s 256 + e) TC + c = copy c of entry e of stage s
        for (int v = wave; v < S * 4 * G::TC; v += 8) {
            const int u = 64 * v + lane, se = u / G::TC;
            const uint4 *src = reinterpret_cast<const uint4 *>(a.tabh[se >> 8]) + (se & 255);
            __builtin_amdgcn_global_load_lds(src, s_tab4 + 64 * v, 16, 0, 0);
        }
    }
    dma_group(0, 0, kb, 0, true);
#pragma unroll
    for (int c = 0; c < G::NS - 1; ++c) dma_group(clampk(kb + c), c, clampk(kb + c + 1), (c + 1) % G::NS, false);

    // code and gain words of this wave's chunks in weight slot sw: d = 8,
    // chunks 4 g + 2 kh and + 1 (two codes, two gains); d = 16, chunk 2 g + kh
    uint32_t cw[NT][S], gw[NT][S];
    auto load_words = [&](int sw) {
        const uint8_t *ws = s_wr + sw * G::WSLOT;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int grp = NT * rs + j, jt = grp >> 2, rit = 16 * (grp & 3) + r16;
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const uint8_t *base = ws + (jt * S + s) * (G::WU * 16);
                if constexpr (D == 8) {
                    cw[j][s] = *reinterpret_cast<const uint16_t *>(base + rit * 16 + 4 * g + 2 * kh);
                    gw[j][s] = *reinterpret_cast<const uint32_t *>(base + 1024 + rit * 32 + 8 * g + 4 * kh);
                } else {
                    cw[j][s] = *reinterpret_cast<const uint16_t *>(base + rit * 16 + 4 * g + 2 * kh);
                    gw[j][s] = *reinterpret_cast<const uint16_t *>(base + 1024 + rit * 16 + 4 * g + 2 * kh);
                }
            }
        }
    };
    // decoder entries of both k-slices: tv[j][u][s] (d = 16: the two halves
    // of the chunk's entry are u = 0, 1; global loads)
    f16x8_t tv[NT][2][S];
    auto load_tables = [&]() {
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int s = 0; s < S; ++s) {
                if constexpr (D == 8) {
#pragma unroll
                    for (int u = 0; u < 2; ++u)
                        tv[j][u][s] = *reinterpret_cast<const f16x8_t *>(
                            s_tab + ((s * 256 + ((cw[j][s] >> (8 * u)) & 0xffu)) * G::TC + (lane & (G::TC - 1))) * 8);
                } else {
                    const f16x8_t *y = reinterpret_cast<const f16x8_t *>(a.tabh[s] + size_t(cw[j][s] & 0xffffu) * 16);
                    tv[j][0][s] = y[0];
                    tv[j][1][s] = y[1];
                }
            }
    };
    // B fragments: bq[j][u] = the 8 bf16 weights of the lane's inputs in
    // k-slice 2 kh + u, each sum_s gain_s * D_s(code_s)[e] as an fp32 fma
    // chain over fp16 gains and fp16 table values, rounded to bf16
    auto decode = [&](u32x4_t (&bq)[NT][2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                float v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = 0.0f;
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    const float gs = f16_bits_to_f32(uint16_t((D == 8) ? (gw[j][s] >> (16 * u)) : gw[j][s]));
#pragma unroll
                    for (int e = 0; e < 8; ++e) v[e] = __builtin_fmaf(gs, float(tv[j][u][s][e]), v[e]);
                }
                bq[j][u] = u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
            }
    };

    u32x4_t bq[NT][2];
    // group -1 has landed (the NS - 1 younger groups may still be in flight)
    if (pw == G::PMAX) wait_vm<(G::NS - 1) * G::PMAX>();
    else wait_vm<(G::NS - 1) * G::PMIN>();
    lds_barrier();
    load_words(0);
    load_tables();
    decode(bq);

    f32x4_t acc[MT][NT];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    int sx = 0;                      // X~ slot of step ks (c % NS)
    int swn = (G::NS > 1) ? 1 : 0;   // weight slot of step ks + 1 ((c + 1) % NS)
    for (int64_t ks = kb; ks < ke; ++ks) {
        if (pw == G::PMAX) wait_vm<(G::NS - 2) * G::PMAX>();
        else wait_vm<(G::NS - 2) * G::PMIN>();
        lds_barrier();
        load_words(swn);
        if constexpr (D == 16) load_tables();  // global: issued before this iteration's DMA
        {
            // group c + NS - 1: X~ slot (c - 1) % NS, weight slot c % NS
            const int slx = (sx == 0) ? G::NS - 1 : sx - 1;
            const int slw = (swn == 0) ? G::NS - 1 : swn - 1;
            dma_group(clampk(ks + G::NS - 1), slx, clampk(ks + G::NS), slw, false);
        }
        if constexpr (D == 8) load_tables();
        const uint8_t *xs = s_xr + sx * G::XSLOT;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            u32x4_t av[MT];
#pragma unroll
            for (int i = 0; i < MT; ++i)
                av[i] = reinterpret_cast<const u32x4_t *>(xs)[((2 * kh + u) * MT + i) * 64 + lane];
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < NT; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av[i]),
                                                                         __builtin_bit_cast(bf16x8_t, bq[j][u]), acc[i][j], 0, 0, 0);
        }
        decode(bq);  // step ks + 1
        sx = (sx + 1 == G::NS) ? 0 : sx + 1;
        swn = (swn + 1 == G::NS) ? 0 : swn + 1;
    }
    // the clamped DMAs past the last step land before the ring is reused
    wait_vm<0>();
    lds_barrier();

    // protected term (split 0, by the kh = 1 waves): X[:, idx] (bf16) times
    // bf16(value(q8) s), the weights of lane row 16 (NT rs + j) + lane % 16 at
    // positions 32 qq + 8 g + e; two slices of 32 positions per round (one
    // with 256-token tiles, whose activations fill the registers), all
    // their loads issued together (stored bytes as one 8-byte word per row;
    // positions past k read as zero)
    if (kh == 1 && z == 0 && a.k > 0) {
        const int64_t kp = q8_pitch(a.k), nq = a.kp32 / 32;
        constexpr int H = (MT > 8) ? 1 : 2;
        for (int64_t q0 = 0; q0 < nq; q0 += H) {
            uint2 qv[H][NT];
            float sc[H][8];
            u32x4_t xv[H][MT];
#pragma unroll
            for (int h = 0; h < H; ++h) {
                const bool live = q0 + h < nq;
                const int64_t p0 = 32 * (q0 + h) + 8 * g;
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    const int64_t row = n0 + 16 * (NT * rs + j) + r16;
                    qv[h][j] = (live && row < a.d_out && p0 < kp) ? *reinterpret_cast<const uint2 *>(a.q8 + row * kp + p0)
                                                                  : make_uint2(0u, 0u);
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) sc[h][e] = (live && p0 + e < a.k) ? a.scale[p0 + e] : 0.0f;
#pragma unroll
                for (int i = 0; i < MT; ++i)
                    xv[h][i] = live ? *reinterpret_cast<const u32x4_t *>(a.Xp + (m0 + 16 * i + r16) * a.kp32 + p0)
                                    : u32x4_t{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int h = 0; h < H; ++h) {
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    float v[8];
                    payload8(qv[h][j], sc[h], v, a.pfmt);
                    const u32x4_t bp = u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                                               pack_bf16x2(v[6], v[7])};
#pragma unroll
                    for (int i = 0; i < MT; ++i)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, xv[h][i]),
                                                                             __builtin_bit_cast(bf16x8_t, bp), acc[i][j], 0, 0, 0);
                }
            }
        }
    }

    // LoRA (finishing split, by the kh = 1 waves): T B^T through the same
    // MFMA. T (fp32) is split exactly into three bf16 parts, hi + mid + lo,
    // whose sum equals T to 2^-24 relative; k-inputs 0..15 of the first
    // product carry hi and 16..31 mid, both against B[:, 0..15] (bf16,
    // exact), the second product lo. Every product of bf16 parts is exact in
    // fp32, so the term is T B^T to within the fp32 accumulation.
    if (kh == 1 && z == a.ksplit - 1 && a.rank > 0) {
        const int q0 = 8 * (g & 1);
        u32x4_t bl[NT], bz[NT];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int64_t n = n0 + 16 * (NT * rs + j) + r16;
            const int64_t nc = (n < a.d_out) ? n : a.d_out - 1;
            float b[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) b[e] = (q0 + e < a.rank) ? bf16_to_f32(a.B[nc * a.rank + q0 + e]) : 0.0f;
            bl[j] = u32x4_t{pack_bf16x2(b[0], b[1]), pack_bf16x2(b[2], b[3]), pack_bf16x2(b[4], b[5]), pack_bf16x2(b[6], b[7])};
            bz[j] = (g < 2) ? bl[j] : u32x4_t{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const float4 *tp = reinterpret_cast<const float4 *>(a.T + (m0 + 16 * i + r16) * BSQ_MAX_LORA_RANK + q0);
            const float4 t0 = tp[0], t1 = tp[1];
            const float tv8[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
            uint32_t hi[4], mid[4], lo[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                hi[e] = pack_bf16x2(tv8[2 * e], tv8[2 * e + 1]);
                const float r0 = tv8[2 * e] - __uint_as_float(hi[e] << 16);
                const float r1 = tv8[2 * e + 1] - __uint_as_float(hi[e] & 0xffff0000u);
                mid[e] = pack_bf16x2(r0, r1);
                lo[e] = pack_bf16x2(r0 - __uint_as_float(mid[e] << 16), r1 - __uint_as_float(mid[e] & 0xffff0000u));
            }
            const uint32_t *p1 = (g < 2) ? hi : mid;
            const u32x4_t a1 = u32x4_t{p1[0], p1[1], p1[2], p1[3]};
            const u32x4_t a2 = u32x4_t{lo[0], lo[1], lo[2], lo[3]};
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a1),
                                                                     __builtin_bit_cast(bf16x8_t, bl[j]), acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a2),
                                                                     __builtin_bit_cast(bf16x8_t, bz[j]), acc[i][j], 0, 0, 0);
            }
        }
    }

    // the kh = 1 half of every row set hands its tile to the kh = 0 half
    // through LDS (the X~ ring, free now), which adds it (kh 0 + kh 1) and
    // puts the block's tile in LDS as fp32 [BM][BN + 4] rows
    f32x4_t *s_red = reinterpret_cast<f32x4_t *>(s_mem);
    if (kh == 1) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) s_red[((rs * MT + i) * NT + j) * 64 + lane] = acc[i][j];
    }
    lds_barrier();
    if (kh == 0) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) acc[i][j] = acc[i][j] + s_red[((rs * MT + i) * NT + j) * 64 + lane];
    }
    lds_barrier();  // the exchange area is free again
    constexpr int OS = G::BN + 4;  // row stride of the staged tile (floats)
    static_assert(size_t(G::BM) * OS * 4 <= G::LDS, "the output tile fits in LDS");
    float *s_out = reinterpret_cast<float *>(s_mem);
    if (kh == 0) {
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) s_out[(16 * i + 4 * g + r) * OS + 16 * (NT * rs + j) + r16] = acc[i][j][r];
    }
    lds_barrier();

    // From here every thread works on 8-output segments of the tile's rows:
    // segment e = token row e / (BN / 8), outputs 8 (e % (BN / 8)) .. + 8.
    constexpr int SEGS = G::BM * (G::BN / 8);
    constexpr int NSEG = (SEGS + 511) / 512;  // segments per thread (t + 512 k)
    if (a.ksplit > 1) {
        // the split's partial tile to part[z] (rows of the padded token
        // range, whole blocks of rows: every element the sum reads is written)
        const int64_t mp = int64_t(gridDim.y) * G::BM;
        float *pz = a.part + (int64_t(z) * mp + m0) * a.np + n0;
#pragma unroll
        for (int k = 0; k < NSEG; ++k) {
            const int e = t + 512 * k;
            if (e >= SEGS) break;
            const int ml = e / (G::BN / 8), nl = 8 * (e % (G::BN / 8));
            float4 *dst = reinterpret_cast<float4 *>(pz + ml * a.np + nl);
            dst[0] = *reinterpret_cast<const float4 *>(s_out + ml * OS + nl);
            dst[1] = *reinterpret_cast<const float4 *>(s_out + ml * OS + nl + 4);
        }
        return;
    }

    // store: one 16-byte store per bf16 segment, two per fp32 segment, when
    // Y allows; element stores at a ragged edge
#pragma unroll
    for (int k = 0; k < NSEG; ++k) {
        const int e = t + 512 * k;
        if (e >= SEGS) break;
        const int ml = e / (G::BN / 8), nl = 8 * (e % (G::BN / 8));
        const int64_t m = m0 + ml, n = n0 + nl;
        if (m >= a.M || n >= a.d_out) continue;
        const float4 lo = *reinterpret_cast<const float4 *>(s_out + ml * OS + nl);
        const float4 hi = *reinterpret_cast<const float4 *>(s_out + ml * OS + nl + 4);
        const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        if (a.y_vec && n + 8 <= a.d_out) {
            if (a.y_bf16) {
                *reinterpret_cast<u32x4_t *>(static_cast<uint16_t *>(a.Y) + m * a.ldy + n) =
                    u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
            } else {
                float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(a.Y) + m * a.ldy + n);
                dst[0] = lo;
                dst[1] = hi;
            }
        } else {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                if (n + c >= a.d_out) break;
                if (a.y_bf16) static_cast<uint16_t *>(a.Y)[m * a.ldy + n + c] = f32_to_bf16(v[c]);
                else static_cast<float *>(a.Y)[m * a.ldy + n + c] = v[c];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Codes of b != d bits per chunk (a codec with a linear encoder): the
// 2^b-entry decoder table does not suit the MFMA paths' decode, so the
// product runs in fp32 over LDS tiles of decoded weights. A workgroup of 256
// threads owns 64 rows x 32 tokens. Per 128-input K step it decodes the
// 64 x 128 weight tile into LDS (each weight the fmaf chain over the stages
// from 0, gain times fp32 table entry, as in decode), converts the X~ tile
// (bf16, protected columns zero, written by gemm_prep) to fp32 in LDS, and
// each thread accumulates 4 rows x 2 tokens. The protected term uses the
// gathered activations and the LoRA term T = X A^T, both from gemm_prep.
// ---------------------------------------------------------------------------
struct GenericGemmArgs {
    const void *codes[BSQ_MAX_STAGES];
    const uint16_t *gains[BSQ_MAX_STAGES];
    const float *tab32[BSQ_MAX_STAGES];
    const int8_t *q8;
    const float *scale;
    const uint16_t *Xt, *Xp, *B;
    const float *T;
    int rank, pfmt, y_bf16;
    int64_t M, d_out, pitch, C, ksteps, Kp, k, kp32, ldy;
    void *Y;
};

template <int D, int B, int S>
__global__ __launch_bounds__(256) void gemm_generic_kernel(const GenericGemmArgs a)
{
    __shared__ float s_w[64][BK + 1];
    __shared__ float s_x[32][BK + 1];
    const int t = threadIdx.x;
    const int64_t n0 = int64_t(blockIdx.x) * 64, m0 = int64_t(blockIdx.y) * 32;
    const int tr = t >> 4, tc = t & 15;  // rows 4 tr .. + 3, tokens 2 tc, 2 tc + 1
    constexpr int CPK = BK / D;          // chunks per K step
    float acc[4][2] = {};
    for (int64_t ks = 0; ks < a.ksteps; ++ks) {
        for (int e = t; e < 64 * CPK; e += 256) {
            const int r = e / CPK, cc = e - r * CPK;
            const int64_t row = n0 + r, c = ks * CPK + cc;
            float v[D];
#pragma unroll
            for (int j = 0; j < D; ++j) v[j] = 0.0f;
            if (row < a.d_out && c < a.C) {
                const int64_t off = tile_index(row, c, a.pitch);
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    const uint32_t code = (B == 8) ? uint32_t(static_cast<const uint8_t *>(a.codes[s])[off])
                                                   : uint32_t(static_cast<const uint16_t *>(a.codes[s])[off]);
                    const float g = f16_bits_to_f32(a.gains[s][off]);
                    const float *y = a.tab32[s] + size_t(code) * D;
#pragma unroll
                    for (int j = 0; j < D; ++j) v[j] = __builtin_fmaf(g, y[j], v[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < D; ++j) s_w[r][cc * D + j] = v[j];
        }
        for (int e = t; e < 32 * BK; e += 256) {
            const int tok = e / BK, col = e - tok * BK;
            const int64_t mt = m0 + tok;
            s_x[tok][col] = (mt < a.M) ? bf16_to_f32(a.Xt[mt * a.Kp + ks * BK + col]) : 0.0f;
        }
        __syncthreads();
#pragma unroll 4
        for (int kk = 0; kk < BK; ++kk) {
            const float x0 = s_x[2 * tc][kk], x1 = s_x[2 * tc + 1][kk];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float w = s_w[4 * tr + i][kk];
                acc[i][0] = __builtin_fmaf(w, x0, acc[i][0]);
                acc[i][1] = __builtin_fmaf(w, x1, acc[i][1]);
            }
        }
        __syncthreads();
    }
    const int64_t kp = q8_pitch(a.k);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = n0 + 4 * tr + i;
        if (row >= a.d_out) continue;
#pragma unroll
        for (int jt = 0; jt < 2; ++jt) {
            const int64_t tok = m0 + 2 * tc + jt;
            if (tok >= a.M) continue;
            float v = acc[i][jt];
            for (int64_t p = 0; p < a.k; ++p)
                v = __builtin_fmaf(payload_to_f32(uint8_t(a.q8[row * kp + p]), a.pfmt) * a.scale[p],
                                   bf16_to_f32(a.Xp[tok * a.kp32 + p]), v);
            for (int r = 0; r < a.rank; ++r)
                v = __builtin_fmaf(bf16_to_f32(a.B[row * a.rank + r]), a.T[tok * BSQ_MAX_LORA_RANK + r], v);
            if (a.y_bf16) static_cast<uint16_t *>(a.Y)[tok * a.ldy + row] = f32_to_bf16(v);
            else static_cast<float *>(a.Y)[tok * a.ldy + row] = v;
        }
    }
}

template <int D, int B>
hipError_t launch_generic_t(int stages, const GenericGemmArgs &g, hipStream_t st)
{
    const dim3 grid(unsigned((g.d_out + 63) / 64), unsigned((g.M + 31) / 32));
    switch (stages) {
    case 1: hipLaunchKernelGGL((gemm_generic_kernel<D, B, 1>), grid, dim3(256), 0, st, g); break;
    case 2: hipLaunchKernelGGL((gemm_generic_kernel<D, B, 2>), grid, dim3(256), 0, st, g); break;
    case 3: hipLaunchKernelGGL((gemm_generic_kernel<D, B, 3>), grid, dim3(256), 0, st, g); break;
    default: hipLaunchKernelGGL((gemm_generic_kernel<D, B, 4>), grid, dim3(256), 0, st, g); break;
    }
    return hipGetLastError();
}

// Launch shape: token tile and rows per block by M, then the K split, then
// the workspace layout.
struct GemmPlan {
    int mt, nt;  // token groups and 64-row groups per block
    int64_t bm, bn, mtiles, nblk, ksteps, ksplit, Mp, Kp, kp32;
    int64_t np;  // d_out padded to whole blocks (partials' row pitch)
    size_t t_off, xt_off, xp_off, part_off, total;
};

GemmPlan gemm_plan(int d, int stages, int64_t d_out, int64_t d_in, int64_t M, int64_t k)
{
    GemmPlan p{};
    // token tiles of 16 tokens up to 16 tokens, for projections of at most
    // 2048 rows up to 64 tokens, and at d = 8 up to 32 tokens (these blocks
    // run three per compute unit, and a block's token tiles share its
    // weights through L2); 64-token tiles up to 64 tokens, and at d = 8 of
    // 64-row blocks (two per compute unit) for projections of at most 4096 x
    // 4096 up to 128 tokens and of at most 2048 rows up to 256 tokens, else
    // 128-token tiles; at d = 16 above 128 tokens one 256-token tile of
    // 64-row blocks, so that each chunk's entry of the 2^16-entry table is
    // gathered once per block rather than once per token tile (at d = 8 the
    // 256-token tile measured slower: its decode is cheap and two ring slots
    // are too few)
    const bool mid8 = d == 8 && M > 64 && d_in <= 4096 && ((M <= 128 && d_out <= 4096) || (M <= 256 && d_out <= 2048));
    p.mt = (M <= 16 || (M <= 64 && d_out <= 2048) || (d == 8 && M <= 32)) ? 1
           : (M <= 64 || mid8)                                          ? 4
           : (d == 16 && M > 128)                                       ? 16
                                                                        : 8;
    // 64-row blocks with 16- and 256-token tiles, at d = 16 with 64-token
    // tiles (two per compute unit), with the 64-token tiles above 64 tokens
    // named above, and at d = 8 up to 64 tokens where both dimensions are at
    // most 4096 and for at most 2048 rows of at most 4096 inputs (twice the
    // blocks, so fewer K splits and a lighter split-K sum; they measured
    // faster there, not on the longer projections); 128-row blocks otherwise
    p.nt = (p.mt == 1 || p.mt == 16 || (d == 16 && p.mt == 4) || mid8 || (d == 8 && d_out <= 4096 && d_in <= 4096 && (M <= 64 || d_out <= 2048))) ? 1 : 2;
    p.bm = 16 * p.mt;
    p.bn = 64 * p.nt;
    p.mtiles = (M + p.bm - 1) / p.bm;
    p.nblk = (d_out + p.bn - 1) / p.bn;
    p.ksteps = (d_in + BK - 1) / BK;
    p.Mp = std::max<int64_t>(p.mtiles, 1) * p.bm;
    p.Kp = p.ksteps * BK;
    p.kp32 = (k + 31) & ~int64_t(31);
    const int64_t tiles = p.nblk * p.mtiles;
    // one workgroup per compute unit (the LDS rings take most of its LDS):
    // split K as far as one round of workgroups over the 256 compute units
    // allows (a second, partial round would double the time), keeping at least
    // 2 K steps per split and at most 8 splits (the partials of all splits
    // are written and read once more: at most 256 tiles' worth, 16 MiB).
    // Blocks that run two or three per compute unit: up to 512 or 768
    // workgroups, with at least 8 K steps per split (shorter splits measured
    // slower), but never fewer splits than the rule above.
    const int64_t nt_ = std::max<int64_t>(tiles, 1);
    int64_t ks = std::min<int64_t>({256 / nt_, p.ksteps / 2, 8});
    const int wpc = gemm_wg_per_cu(d, stages, int(p.mt), int(p.nt));
    if (wpc > 1) ks = std::max(ks, std::min<int64_t>({256 * wpc / nt_, p.ksteps / 8, 8}));
    p.ksplit = std::max<int64_t>(ks, 1);
    p.t_off = size_t(GEMM_HDR);
    p.xt_off = p.t_off + align256(size_t(p.Mp) * BSQ_MAX_LORA_RANK * 4);
    p.xp_off = p.xt_off + align256(size_t(p.Mp) * size_t(p.Kp) * 2);
    p.part_off = p.xp_off + align256(size_t(p.Mp) * size_t(std::max<int64_t>(p.kp32, 32)) * 2);
    p.np = p.nblk * p.bn;
    p.total = p.part_off + ((p.ksplit > 1) ? size_t(p.ksplit) * size_t(p.Mp) * size_t(p.np) * 4 : 0);
    return p;
}

// Split-K sum: one thread per 8-output segment of Y, the partials added in
// split order (z = 0, 1, ...), stored as the tiled kernel stores. KS is the
// split count, so that all of a thread's loads are issued before the first
// add (a loop over a run-time count waited for each split's loads in turn).
template <int KS>
__global__ __launch_bounds__(256) void gemm_splitk_sum(const GemmArgs a, int64_t mp)
{
    const int64_t nseg = (a.d_out + 7) / 8;
    const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (e >= a.M * nseg) return;
    const int64_t m = e / nseg, n = 8 * (e - m * nseg);
    const float *src = a.part + m * a.np + n;
    float4 l[KS], h[KS];
#pragma unroll
    for (int z = 0; z < KS; ++z) {
        const float4 *pz = reinterpret_cast<const float4 *>(src + int64_t(z) * mp * a.np);
        l[z] = pz[0];
        h[z] = pz[1];
    }
    float4 lo = l[0], hi = h[0];
#pragma unroll
    for (int z = 1; z < KS; ++z) {
        lo.x += l[z].x; lo.y += l[z].y; lo.z += l[z].z; lo.w += l[z].w;
        hi.x += h[z].x; hi.y += h[z].y; hi.z += h[z].z; hi.w += h[z].w;
    }
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    if (a.y_vec && n + 8 <= a.d_out) {
        if (a.y_bf16) {
            *reinterpret_cast<u32x4_t *>(static_cast<uint16_t *>(a.Y) + m * a.ldy + n) =
                u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
        } else {
            float4 *dst = reinterpret_cast<float4 *>(static_cast<float *>(a.Y) + m * a.ldy + n);
            dst[0] = lo;
            dst[1] = hi;
        }
    } else {
        for (int c = 0; c < 8; ++c) {
            if (n + c >= a.d_out) break;
            if (a.y_bf16) static_cast<uint16_t *>(a.Y)[m * a.ldy + n + c] = f32_to_bf16(v[c]);
            else static_cast<float *>(a.Y)[m * a.ldy + n + c] = v[c];
        }
    }
}

template <int D, int S, int MT, int NT>
hipError_t launch_main(const GemmArgs &a, const GemmPlan &p, hipStream_t st)
{
    using G = GemmShape<D, S, MT, NT>;
    static bool lds_set = false;  // the LDS rings exceed the default dynamic LDS limit
    if (!lds_set) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&gemm_kernel<D, S, MT, NT>),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, int(G::LDS));
        if (e != hipSuccess) return e;
        lds_set = true;
    }
    const dim3 grid = dim3(unsigned(p.nblk), unsigned(p.mtiles), unsigned(p.ksplit));
    hipLaunchKernelGGL((gemm_kernel<D, S, MT, NT>), grid, dim3(512), G::LDS, st, a);
    if (p.ksplit > 1) {
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t segs = a.M * ((a.d_out + 7) / 8);
        const dim3 sg(unsigned((segs + 255) / 256));
        switch (p.ksplit) {
        case 2: hipLaunchKernelGGL(gemm_splitk_sum<2>, sg, dim3(256), 0, st, a, p.Mp); break;
        case 3: hipLaunchKernelGGL(gemm_splitk_sum<3>, sg, dim3(256), 0, st, a, p.Mp); break;
        case 4: hipLaunchKernelGGL(gemm_splitk_sum<4>, sg, dim3(256), 0, st, a, p.Mp); break;
        case 5: hipLaunchKernelGGL(gemm_splitk_sum<5>, sg, dim3(256), 0, st, a, p.Mp); break;
        case 6: hipLaunchKernelGGL(gemm_splitk_sum<6>, sg, dim3(256), 0, st, a, p.Mp); break;
        case 7: hipLaunchKernelGGL(gemm_splitk_sum<7>, sg, dim3(256), 0, st, a, p.Mp); break;
        default: hipLaunchKernelGGL(gemm_splitk_sum<8>, sg, dim3(256), 0, st, a, p.Mp); break;
        }
    }
    return hipGetLastError();
}

template <int D, int S>
hipError_t launch_gemm_t(const GemmArgs &a, const GemmPlan &p, hipStream_t st)
{
    // the shapes gemm_plan chooses, and only those
    if constexpr (D == 8) {
        if (p.mt == 1) return launch_main<D, S, 1, 1>(a, p, st);
        if (p.mt == 4) return (p.nt == 1) ? launch_main<D, S, 4, 1>(a, p, st) : launch_main<D, S, 4, 2>(a, p, st);
        return (p.nt == 1) ? launch_main<D, S, 8, 1>(a, p, st) : launch_main<D, S, 8, 2>(a, p, st);
    } else {
        if (p.mt == 1) return launch_main<D, S, 1, 1>(a, p, st);
        if (p.mt == 4) return launch_main<D, S, 4, 1>(a, p, st);
        if (p.mt == 16) return launch_main<D, S, 16, 1>(a, p, st);
        return launch_main<D, S, 8, 2>(a, p, st);
    }
}

}  // namespace

const float *gemm_lora_t(const void *ws)
{
    return reinterpret_cast<const float *>(static_cast<const char *>(ws) + GEMM_HDR);
}

size_t gemm_ws_bytes(const bsq_config &cfg, int64_t d_out, int64_t d_in, int64_t M)
{
    const int64_t k = cfg.protect_num ? (d_in * cfg.protect_num + cfg.protect_den - 1) / cfg.protect_den : 0;
    return gemm_plan(cfg.d, cfg.stages, d_out, d_in, M, k).total;
}

hipError_t launch_gemm(const bsq_config &cfg, const void *codec, const bsq_layer &L, const bsq_lora *lora,
                       const void *X, int64_t M, int64_t ldx, void *Y, int y_dtype, int64_t ldy, void *ws,
                       int32_t *err, hipStream_t st)
{
    if (M == 0 || L.d_out == 0) return hipSuccess;
    const GemmPlan p = gemm_plan(cfg.d, cfg.stages, L.d_out, L.d_in, M, L.k);
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
    {
        const int64_t es = a.y_bf16 ? 2 : 4;
        a.y_vec = (reinterpret_cast<uintptr_t>(Y) % 16 == 0) && ((ldy * es) % 16 == 0);
    }
    a.rank = 0;
    a.ksplit = int(p.ksplit);
    a.part = reinterpret_cast<float *>(wb + p.part_off);
    a.np = p.np;
    (void)err;  // (no block waits for another: there is nothing to report)
    a.pfmt = cfg.protect_format;

    PrepArgs pa{};
    pa.X = static_cast<const uint16_t *>(X);
    pa.ldx = ldx;
    pa.M = M;
    pa.d_in = L.d_in;
    pa.Kp = p.Kp;
    pa.k = L.k;
    pa.kp32 = p.kp32;
    pa.idx = L.prot_idx;
    pa.bits = L.prot_bits;
    pa.Xt = reinterpret_cast<uint16_t *>(wb + p.xt_off);
    pa.Xp = reinterpret_cast<uint16_t *>(wb + p.xp_off);
    pa.T = reinterpret_cast<float *>(wb + p.t_off);
    if (lora && lora->rank > 0) {
        a.rank = lora->rank;
        a.B = lora->B;
        pa.A = lora->A;
        pa.rank = lora->rank;
    }
    // per token row: the X~ column blocks, the gather, then one block per LoRA rank index
    hipLaunchKernelGGL(gemm_prep, dim3(unsigned(p.Mp), unsigned((p.Kp + PREP_COLS - 1) / PREP_COLS + 1 + pa.rank)),
                       dim3(256), 0, st, pa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    const int S = cfg.stages;
    if (cfg.b != cfg.d) {
        GenericGemmArgs g{};
        const char *cb2 = static_cast<const char *>(codec);
        for (int s = 0; s < S; ++s) {
            g.codes[s] = L.codes[s];
            g.gains[s] = L.gains[s];
            g.tab32[s] = reinterpret_cast<const float *>(cb2 + codec_tab32_offset(cfg, s));
        }
        g.q8 = L.prot_q8;
        g.scale = L.prot_scale;
        g.Xt = a.Xt;
        g.Xp = a.Xp;
        g.T = a.T;
        g.B = a.B;
        g.rank = a.rank;
        g.pfmt = cfg.protect_format;
        g.y_bf16 = a.y_bf16;
        g.M = M;
        g.d_out = L.d_out;
        g.pitch = L.pitch;
        g.C = L.d_in / cfg.d;
        g.ksteps = p.ksteps;
        g.Kp = p.Kp;
        g.k = L.k;
        g.kp32 = p.kp32;
        g.ldy = ldy;
        g.Y = Y;
        return (cfg.d == 8) ? launch_generic_t<8, 16>(S, g, st) : launch_generic_t<16, 8>(S, g, st);
    }
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
