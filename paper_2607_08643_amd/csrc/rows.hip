// Protected output rows (eq. protected_8bit_scatter applied to row slices:
// the output-channel axis of the protection-axis ablation, Section IV-D, and
// the gate/up side of eq. mlp_coupled_protection). The coded rows go through
// the streaming decode/GEMV/GEMM kernels, where a protected row's code 0 and
// gain +0 make its BSQ term zero; these kernels then write every protected
// row of the result from its protected payload (value(q8) per the format,
// payload_to_f32), on the same stream:
//   decode  W_hat[idx_p, j] = value(q8[p][j]) * scale_p        (fp32 product)
//   GEMV    y[idx_p]        = scale_p <value(q8[p]), x> + B[idx_p] . (A x)
//   GEMM    Y[t][idx_p]     = scale_p <value(q8[p]), X[t]> + B[idx_p] . T[t]
// (T = X A^T, fp32, left in the GEMM workspace by its activation prep).
// All three are small side launches: k = ceil(rho * d_out) rows.
#include "bsq_internal.h"

namespace bsq {

namespace {

template <bool BF16OUT>
__global__ __launch_bounds__(256) void decode_rows_kernel(const int32_t *__restrict__ idx,
                                                          const int8_t *__restrict__ q8,
                                                          const float *__restrict__ scale, int64_t d_out,
                                                          int64_t d_in, int64_t k, int fmt, void *__restrict__ out)
{
    const int64_t p = blockIdx.x, m = blockIdx.y;
    const int64_t row = idx[m * k + p];
    const float s = scale[m * k + p];
    const int8_t *q = q8 + (m * k + p) * q8_pitch(d_in);
    const int64_t base = (m * d_out + row) * d_in;
    for (int64_t j = threadIdx.x; j < d_in; j += 256) {
        const float v = payload_to_f32(uint8_t(q[j]), fmt) * s;
        if constexpr (BF16OUT) static_cast<uint16_t *>(out)[base + j] = f32_to_bf16(v);
        else static_cast<float *>(out)[base + j] = v;
    }
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

struct RowsGemvArgs {
    const int32_t *idx[BSQ_MAX_GROUP];
    const int8_t *q8[BSQ_MAX_GROUP];
    const float *scale[BSQ_MAX_GROUP];
    const uint16_t *A[BSQ_MAX_GROUP];  // LoRA A [rank][d_in] or null
    const uint16_t *B[BSQ_MAX_GROUP];  // LoRA B [d_out][rank]
    void *y[BSQ_MAX_GROUP];
    int64_t k[BSQ_MAX_GROUP];
    int rank[BSQ_MAX_GROUP];
    const void *x;
    int64_t d_in;
    int x_bf16, y_bf16, pfmt;
};

// One block per (protected row p, matrix m of the group). Each thread sums
// its strided columns of the int8 row and of the rank LoRA rows against x;
// the block then reduces the 1 + rank partial sums.
__global__ __launch_bounds__(256) void gemv_rows_kernel(const RowsGemvArgs a)
{
    __shared__ float red[4][1 + BSQ_MAX_LORA_RANK];
    const int m = blockIdx.y;
    const int64_t p = blockIdx.x;
    if (p >= a.k[m]) return;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int rank = a.rank[m];
    const int8_t *q = a.q8[m] + p * q8_pitch(a.d_in);
    const uint16_t *A = a.A[m];
    float acc = 0.0f, tr[BSQ_MAX_LORA_RANK];
#pragma unroll
    for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r) tr[r] = 0.0f;
    for (int64_t j = t; j < a.d_in; j += 256) {
        const float xv = a.x_bf16 ? bf16_to_f32(static_cast<const uint16_t *>(a.x)[j])
                                  : static_cast<const float *>(a.x)[j];
        acc += payload_to_f32(uint8_t(q[j]), a.pfmt) * xv;
#pragma unroll
        for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r)
            if (r < rank) tr[r] += bf16_to_f32(A[r * a.d_in + j]) * xv;
    }
    acc = wave_sum(acc);
#pragma unroll
    for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r)
        if (r < rank) tr[r] = wave_sum(tr[r]);
    if (lane == 0) {
        red[wave][0] = acc;
#pragma unroll
        for (int r = 0; r < BSQ_MAX_LORA_RANK; ++r) red[wave][1 + r] = tr[r];
    }
    __syncthreads();
    if (t != 0) return;
    const int64_t row = a.idx[m][p];
    float dot = 0.0f, lora = 0.0f;
    for (int w = 0; w < 4; ++w) dot += red[w][0];
    for (int r = 0; r < rank; ++r) {
        float tv = 0.0f;
        for (int w = 0; w < 4; ++w) tv += red[w][1 + r];
        lora += bf16_to_f32(a.B[m][row * rank + r]) * tv;
    }
    const float v = a.scale[m][p] * dot + lora;
    if (a.y_bf16) static_cast<uint16_t *>(a.y[m])[row] = f32_to_bf16(v);
    else static_cast<float *>(a.y[m])[row] = v;
}

struct RowsGemmArgs {
    const int32_t *idx;
    const int8_t *q8;
    const float *scale;
    const uint16_t *B;  // LoRA B [d_out][rank] or null
    const float *T;     // X A^T [>= M][BSQ_MAX_LORA_RANK]
    const uint16_t *X;  // [M][ldx] bf16
    void *Y;            // [M][ldy]
    int64_t M, ldx, ldy, d_in, k;
    int rank, y_bf16, pfmt;
};

// One block per (protected row p, 4 tokens); wave w takes token 4 by + w and
// its lanes stride the row.
__global__ __launch_bounds__(256) void gemm_rows_kernel(const RowsGemmArgs a)
{
    const int64_t p = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int64_t tok = int64_t(blockIdx.y) * 4 + (threadIdx.x >> 6);
    if (tok >= a.M) return;
    const int8_t *q = a.q8 + p * q8_pitch(a.d_in);
    const uint16_t *xr = a.X + tok * a.ldx;
    float acc = 0.0f;
    for (int64_t j = lane; j < a.d_in; j += 64) acc += payload_to_f32(uint8_t(q[j]), a.pfmt) * bf16_to_f32(xr[j]);
    acc = wave_sum(acc);
    if (lane != 0) return;
    const int64_t row = a.idx[p];
    float lora = 0.0f;
    for (int r = 0; r < a.rank; ++r) lora += bf16_to_f32(a.B[row * a.rank + r]) * a.T[tok * BSQ_MAX_LORA_RANK + r];
    const float v = a.scale[p] * acc + lora;
    if (a.y_bf16) static_cast<uint16_t *>(a.Y)[tok * a.ldy + row] = f32_to_bf16(v);
    else static_cast<float *>(a.Y)[tok * a.ldy + row] = v;
}

}  // namespace

hipError_t launch_decode_rows(const bsq_layer &L, int fmt, void *w_hat, int out_dtype, hipStream_t st)
{
    if (L.k == 0 || L.d_in == 0 || L.n_mats == 0) return hipSuccess;
    const dim3 grid{unsigned(L.k), unsigned(L.n_mats)};
    if (out_dtype == BSQ_BF16)
        hipLaunchKernelGGL(decode_rows_kernel<true>, grid, dim3(256), 0, st, L.prot_idx, L.prot_q8, L.prot_scale,
                           L.d_out, L.d_in, L.k, fmt, w_hat);
    else
        hipLaunchKernelGGL(decode_rows_kernel<false>, grid, dim3(256), 0, st, L.prot_idx, L.prot_q8, L.prot_scale,
                           L.d_out, L.d_in, L.k, fmt, w_hat);
    return hipGetLastError();
}

hipError_t launch_gemv_rows(int n, const bsq_layer *layers, int fmt, const bsq_lora *loras, const void *x,
                            int x_dtype, void *const *y, int y_dtype, hipStream_t st)
{
    RowsGemvArgs a{};
    int64_t kmax = 0;
    for (int m = 0; m < n; ++m) {
        const bsq_layer &L = layers[m];
        a.idx[m] = L.prot_idx;
        a.q8[m] = L.prot_q8;
        a.scale[m] = L.prot_scale;
        a.k[m] = L.k;
        a.y[m] = y[m];
        if (loras && loras[m].rank > 0) {
            a.A[m] = loras[m].A;
            a.B[m] = loras[m].B;
            a.rank[m] = loras[m].rank;
        }
        kmax = L.k > kmax ? L.k : kmax;
    }
    if (kmax == 0) return hipSuccess;
    a.x = x;
    a.d_in = layers[0].d_in;
    a.x_bf16 = (x_dtype == BSQ_BF16);
    a.y_bf16 = (y_dtype == BSQ_BF16);
    a.pfmt = fmt;
    hipLaunchKernelGGL(gemv_rows_kernel, dim3(unsigned(kmax), unsigned(n)), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_gemm_rows(const bsq_layer &L, int fmt, const bsq_lora *lora, const void *X, int64_t M,
                            int64_t ldx, void *Y, int y_dtype, int64_t ldy, const float *T, hipStream_t st)
{
    if (L.k == 0 || M == 0) return hipSuccess;
    RowsGemmArgs a{};
    a.idx = L.prot_idx;
    a.q8 = L.prot_q8;
    a.scale = L.prot_scale;
    a.T = T;
    a.X = static_cast<const uint16_t *>(X);
    a.Y = Y;
    a.M = M;
    a.ldx = ldx;
    a.ldy = ldy;
    a.d_in = L.d_in;
    a.k = L.k;
    a.y_bf16 = (y_dtype == BSQ_BF16);
    a.pfmt = fmt;
    if (lora && lora->rank > 0) {
        a.B = lora->B;
        a.rank = lora->rank;
    }
    hipLaunchKernelGGL(gemm_rows_kernel, dim3(unsigned(L.k), unsigned((M + 3) / 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace bsq
