// Codec training (Section III-C; eq. codec_loss, eq. codec_loss_terms) for
// one stage codec: the linear encoder z = E x, the sphere map u = z / ||z||,
// sign binarisation with the straight-through estimator, the symmetric
// decoder x_hat = W2 relu(W1 q + b1) + b2, and the loss
//   L = L_rec + lambda_c L_com + lambda_e L_ent
// over a mini-batch of chunks gathered from a category's stacked layers
// (Section III-G, category-batched codec optimisation), then Adam.
//
// Parameters are one fp32 vector theta = E [b][d] | W1 [h][b] | b1 [h] |
// W2 [d][h] | b2 [d]. Every reduction runs in a fixed order, so a step gives
// the same bits on every run:
//   1. train_bits_kernel: per chunk z, u and the bit probabilities
//      s_ij = sigma(2 tau u_ij / sqrt(b)); per block the sums of s and of the
//      per-chunk entropies;
//   2. train_bar_kernel: s_bar_j (the batch's mean bit probability) and the
//      batch entropy;
//   3. train_back_kernel: per chunk the decoder's forward and backward and
//      the straight-through gradient into u and z; writes the per-chunk
//      vectors the parameter gradient needs and per-block loss sums;
//   4. train_param_kernel: each parameter's gradient as a sum over the
//      chunks of one group (G groups), then train_sum_kernel adds the groups
//      and the loss partials in order;
//   5. train_adam_kernel: one Adam step.
#include "bsq_internal.h"

namespace bsq {
namespace {

constexpr int TB = 256;        // threads per block in the per-chunk kernels
constexpr int PG = 512;        // chunk groups of the parameter reduction

struct TrainArgs {
    const void *x;             // chunks [n_total][d], fp32 or bf16
    int x_bf16;
    const int64_t *idx;        // batch chunk indices [n], or null (chunks 0 .. n-1)
    int64_t n, n_total;
    int32_t *err;              // device error word (an index out of range), or null
    int d, b, h;
    const float *theta;
    float lambda_c, lambda_e, gamma, tau, cscale;
    float *s_part;             // [nblk][b] sums of s per block
    float *h_part;             // [nblk] sums of per-chunk entropies per block
    float *sbar;               // [b]
    float *bar_ent;            // [1] sum_j H(s_bar_j)
    float *l_part;             // [nblk][2] sums of ||x_hat - x||^2 and ||u - q||^2 per block
    float *rec;                // [n][R] per-chunk vectors
    int64_t R;
    float *g_part;             // [PG][P]
    float *grad;               // [P]
    float *loss;               // [4]: L, L_rec, L_com, L_ent
    int64_t P, nblk;
};

__device__ __forceinline__ float load_chunk_elem(const TrainArgs &a, int64_t c, int j)
{
    const int64_t e = c * a.d + j;
    return a.x_bf16 ? bf16_to_f32(static_cast<const uint16_t *>(a.x)[e]) : static_cast<const float *>(a.x)[e];
}

__device__ __forceinline__ float entropy2(float s) { return -(s * logf(s) + (1.0f - s) * logf(1.0f - s)); }

// z = E x (fmaf chain from +0, j in order), ||z||, u, and the code (bit m =
// z_m >= 0, the decision the oracle takes in the same chain)
template <int D, int B>
__device__ __forceinline__ void encode_chunk(const TrainArgs &a, const float *E, const float (&x)[D], float (&u)[B],
                                             float &nz, uint32_t &code)
{
    float z[B];
    float ss = 0.0f;
    code = 0;
#pragma unroll
    for (int m = 0; m < B; ++m) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < D; ++j) acc = __builtin_fmaf(E[m * D + j], x[j], acc);
        z[m] = acc;
        code |= (acc >= 0.0f ? 1u : 0u) << m;
        ss = __builtin_fmaf(acc, acc, ss);
    }
    nz = __builtin_sqrtf(ss);
    const float inv = (nz > 0.0f) ? 1.0f / nz : 0.0f;
#pragma unroll
    for (int m = 0; m < B; ++m) u[m] = z[m] * inv;
}

template <int D>
__device__ __forceinline__ void load_x_chunk(const TrainArgs &a, int64_t i, float (&x)[D])
{
    int64_t c = a.idx ? a.idx[i] : i;
    if (c < 0 || c >= a.n_total) {  // reported, and read as chunk 0
        if (a.err) atomicOr(a.err, int32_t(BSQ_DEVERR_BAD_SET));
        c = 0;
    }
#pragma unroll
    for (int j = 0; j < D; ++j) x[j] = load_chunk_elem(a, c, j);
}

// block sum of v in LDS, fixed order (tree over the 256 threads)
__device__ __forceinline__ float block_sum(float v, float *red)
{
    const int t = threadIdx.x;
    red[t] = v;
    __syncthreads();
#pragma unroll
    for (int o = TB / 2; o > 0; o >>= 1) {
        if (t < o) red[t] = red[t] + red[t + o];
        __syncthreads();
    }
    const float r = red[0];
    __syncthreads();
    return r;
}

template <int D, int B>
__global__ __launch_bounds__(TB) void train_bits_kernel(const TrainArgs a)
{
    __shared__ float s_E[B * D];
    __shared__ float red[TB];
    for (int e = threadIdx.x; e < B * D; e += TB) s_E[e] = a.theta[e];
    __syncthreads();
    const int64_t i = int64_t(blockIdx.x) * TB + threadIdx.x;
    float s[B];
    float hsum = 0.0f;
#pragma unroll
    for (int m = 0; m < B; ++m) s[m] = 0.0f;
    if (i < a.n) {
        float x[D], u[B], nz;
        uint32_t code;
        load_x_chunk<D>(a, i, x);
        encode_chunk<D, B>(a, s_E, x, u, nz, code);
        const float k = 2.0f * a.tau * a.cscale;
#pragma unroll
        for (int m = 0; m < B; ++m) {
            s[m] = 1.0f / (1.0f + expf(-k * u[m]));
            hsum += entropy2(s[m]);
        }
    }
#pragma unroll
    for (int m = 0; m < B; ++m) {
        const float v = block_sum(s[m], red);
        if (threadIdx.x == 0) a.s_part[int64_t(blockIdx.x) * B + m] = v;
    }
    const float hv = block_sum(hsum, red);
    if (threadIdx.x == 0) a.h_part[blockIdx.x] = hv;
}

// one block: s_bar_j = sum over the blocks in order / n, and sum_j H(s_bar_j)
__global__ __launch_bounds__(64) void train_bar_kernel(const TrainArgs a)
{
    const int m = threadIdx.x;
    if (m < a.b) {
        float acc = 0.0f;
        for (int64_t k = 0; k < a.nblk; ++k) acc += a.s_part[k * a.b + m];
        a.sbar[m] = acc / float(a.n);
    }
    __syncthreads();
    if (m == 0) {
        float e = 0.0f;
        for (int j = 0; j < a.b; ++j) e += entropy2(a.sbar[j]);
        a.bar_ent[0] = e;
    }
}

// Per chunk: the decoder's forward and backward and the straight-through
// gradient into z. The record of chunk i is
//   [dx_hat (D) | a (h) | dpre (h) | q (B) | dz (B) | x (D)].
template <int D, int B>
__global__ __launch_bounds__(TB) void train_back_kernel(const TrainArgs a)
{
    extern __shared__ float s_theta[];  // the whole parameter vector
    __shared__ float red[TB];
    __shared__ float s_bar[16];
    for (int64_t e = threadIdx.x; e < a.P; e += TB) s_theta[e] = a.theta[e];
    if (threadIdx.x < B) s_bar[threadIdx.x] = a.sbar[threadIdx.x];
    __syncthreads();
    const int h = a.h;
    const float *E = s_theta, *W1 = E + B * D, *b1 = W1 + h * B, *W2 = b1 + h, *b2 = W2 + D * h;
    const int64_t i = int64_t(blockIdx.x) * TB + threadIdx.x;
    float lrec = 0.0f, lcom = 0.0f;
    if (i < a.n) {
        const float inv_n = 1.0f / float(a.n);
        float x[D], u[B], nz;
        uint32_t code;
        load_x_chunk<D>(a, i, x);
        encode_chunk<D, B>(a, E, x, u, nz, code);
        float q[B];
#pragma unroll
        for (int m = 0; m < B; ++m) q[m] = ((code >> m) & 1u) ? a.cscale : -a.cscale;
        // decoder forward: pre_k = fmaf chain from b1_k over j (the decision
        // chain of the oracle), a = relu(pre), x_hat = W2 a + b2
        float act[BSQ_MAX_HIDDEN];
        for (int k = 0; k < h; ++k) {
            float acc = b1[k];
#pragma unroll
            for (int j = 0; j < B; ++j) acc = __builtin_fmaf(W1[k * B + j], q[j], acc);
            act[k] = (acc > 0.0f) ? acc : 0.0f;
        }
        float dxh[D];
#pragma unroll
        for (int mm = 0; mm < D; ++mm) {
            float acc = b2[mm];
            for (int k = 0; k < h; ++k) acc = __builtin_fmaf(W2[mm * h + k], act[k], acc);
            const float df = acc - x[mm];
            lrec = __builtin_fmaf(df, df, lrec);
            dxh[mm] = 2.0f * df * inv_n;
        }
        float *r = a.rec + i * a.R;
        float du[B];
#pragma unroll
        for (int j = 0; j < B; ++j) du[j] = 0.0f;
        for (int k = 0; k < h; ++k) {
            float g = 0.0f;
            if (act[k] > 0.0f) {
#pragma unroll
                for (int mm = 0; mm < D; ++mm) g = __builtin_fmaf(W2[mm * h + k], dxh[mm], g);
            }
            r[D + k] = act[k];
            r[D + h + k] = g;  // dpre
#pragma unroll
            for (int j = 0; j < B; ++j) du[j] = __builtin_fmaf(W1[k * B + j], g, du[j]);
        }
        // commitment and entropy terms into u
        const float k2 = 2.0f * a.tau * a.cscale;
        float udu = 0.0f;
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const float dq = u[j] - q[j];
            lcom = __builtin_fmaf(dq, dq, lcom);
            const float t = k2 * u[j];
            const float s = 1.0f / (1.0f + expf(-t));
            const float sd = s * (1.0f - s);
            const float dt = (-t * sd - a.gamma * logf((1.0f - s_bar[j]) / s_bar[j]) * sd) * inv_n;
            du[j] += a.lambda_c * 2.0f * dq * inv_n + a.lambda_e * dt * k2;
            udu = __builtin_fmaf(u[j], du[j], udu);
        }
        const float inz = (nz > 0.0f) ? 1.0f / nz : 0.0f;
#pragma unroll
        for (int mm = 0; mm < D; ++mm) {
            r[mm] = dxh[mm];
            r[D + 2 * h + B + B + mm] = x[mm];
        }
#pragma unroll
        for (int j = 0; j < B; ++j) {
            r[D + 2 * h + j] = q[j];
            r[D + 2 * h + B + j] = (du[j] - u[j] * udu) * inz;
        }
    }
    const float s1 = block_sum(lrec, red);
    const float s2 = block_sum(lcom, red);
    if (threadIdx.x == 0) {
        a.l_part[int64_t(blockIdx.x) * 2] = s1;
        a.l_part[int64_t(blockIdx.x) * 2 + 1] = s2;
    }
}

// The two record offsets whose product is parameter p's term (-1: the
// factor 1), from the packed layout of theta.
__device__ __forceinline__ void param_factors(const TrainArgs &a, int64_t p, int64_t &o1, int64_t &o2)
{
    const int D = a.d, B = a.b, h = a.h;
    const int64_t oa = D, odp = D + h, oq = D + 2 * h, odz = D + 2 * h + B, ox = D + 2 * h + 2 * B;
    if (p < B * D) {                       // E[m][j]: dz_m x_j
        o1 = odz + p / D;
        o2 = ox + p % D;
        return;
    }
    p -= B * D;
    if (p < int64_t(h) * B) {              // W1[k][j]: dpre_k q_j
        o1 = odp + p / B;
        o2 = oq + p % B;
        return;
    }
    p -= int64_t(h) * B;
    if (p < h) {                           // b1[k]: dpre_k
        o1 = odp + p;
        o2 = -1;
        return;
    }
    p -= h;
    if (p < int64_t(D) * h) {              // W2[m][k]: dx_hat_m a_k
        o1 = p / h;
        o2 = oa + p % h;
        return;
    }
    p -= int64_t(D) * h;                   // b2[m]: dx_hat_m
    o1 = p;
    o2 = -1;
}

// block g sums its chunk range for every parameter (threads stride the
// parameters), chunks in order
__global__ __launch_bounds__(TB) void train_param_kernel(const TrainArgs a)
{
    const int64_t g = blockIdx.x;
    const int64_t c0 = a.n * g / PG, c1 = a.n * (g + 1) / PG;
    for (int64_t p = threadIdx.x; p < a.P; p += TB) {
        int64_t o1, o2;
        param_factors(a, p, o1, o2);
        float acc = 0.0f;
        for (int64_t i = c0; i < c1; ++i) {
            const float *r = a.rec + i * a.R;
            acc = (o2 < 0) ? acc + r[o1] : __builtin_fmaf(r[o1], r[o2], acc);
        }
        a.g_part[g * a.P + p] = acc;
    }
}

// the groups' partial gradients added in order; block 0 also the loss
__global__ __launch_bounds__(TB) void train_sum_kernel(const TrainArgs a)
{
    const int64_t p = int64_t(blockIdx.x) * TB + threadIdx.x;
    if (p < a.P) {
        float acc = 0.0f;
        for (int g = 0; g < PG; ++g) acc += a.g_part[int64_t(g) * a.P + p];
        a.grad[p] = acc;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        float lr = 0.0f, lc = 0.0f, he = 0.0f;
        for (int64_t k = 0; k < a.nblk; ++k) {
            lr += a.l_part[2 * k];
            lc += a.l_part[2 * k + 1];
            he += a.h_part[k];
        }
        const float inv_n = 1.0f / float(a.n);
        const float L_rec = lr * inv_n, L_com = lc * inv_n, L_ent = he * inv_n - a.gamma * a.bar_ent[0];
        a.loss[0] = L_rec + a.lambda_c * L_com + a.lambda_e * L_ent;
        a.loss[1] = L_rec;
        a.loss[2] = L_com;
        a.loss[3] = L_ent;
    }
}

struct AdamArgs {
    float *theta, *m, *v;
    const float *grad;
    int64_t P;
    float lr, beta1, beta2, eps, bc1, bc2;  // bc = 1 - beta^step
};

__global__ __launch_bounds__(TB) void train_adam_kernel(const AdamArgs a)
{
    const int64_t p = int64_t(blockIdx.x) * TB + threadIdx.x;
    if (p >= a.P) return;
    const float g = a.grad[p];
    const float m = a.beta1 * a.m[p] + (1.0f - a.beta1) * g;
    const float v = a.beta2 * a.v[p] + (1.0f - a.beta2) * g * g;
    a.m[p] = m;
    a.v[p] = v;
    a.theta[p] = a.theta[p] - a.lr * (m / a.bc1) / (__builtin_sqrtf(v / a.bc2) + a.eps);
}

template <int D, int B>
hipError_t launch_train_t(const TrainArgs &a, hipStream_t st)
{
    const dim3 grid(unsigned(a.nblk));
    hipLaunchKernelGGL((train_bits_kernel<D, B>), grid, dim3(TB), 0, st, a);
    hipLaunchKernelGGL(train_bar_kernel, dim3(1), dim3(64), 0, st, a);
    hipLaunchKernelGGL((train_back_kernel<D, B>), grid, dim3(TB), size_t(a.P) * 4, st, a);
    hipLaunchKernelGGL(train_param_kernel, dim3(PG), dim3(TB), 0, st, a);
    hipLaunchKernelGGL(train_sum_kernel, dim3(unsigned((a.P + TB - 1) / TB)), dim3(TB), 0, st, a);
    return hipGetLastError();
}

}  // namespace

int64_t train_param_count(const bsq_config &cfg)
{
    const int64_t d = cfg.d, b = cfg.b, h = cfg.hidden;
    return b * d + h * b + h + d * h + d;
}

int64_t train_record_floats(const bsq_config &cfg) { return 2 * cfg.d + 2 * int64_t(cfg.hidden) + 2 * cfg.b; }

size_t train_ws_bytes(const bsq_config &cfg, int64_t n)
{
    const int64_t nblk = (n + TB - 1) / TB, P = train_param_count(cfg);
    return align256(size_t(nblk) * cfg.b * 4) + align256(size_t(nblk) * 4) + 256 + 256 + align256(size_t(nblk) * 8) +
           align256(size_t(n) * train_record_floats(cfg) * 4) + align256(size_t(PG) * P * 4);
}

hipError_t launch_train_grad(const bsq_config &cfg, const bsq_train_hparams &hp, const void *x, int x_dtype,
                             int64_t n_total, const int64_t *idx, int64_t n, const float *theta, float *grad,
                             float *loss, int32_t *err, void *ws, hipStream_t st)
{
    TrainArgs a{};
    a.x = x;
    a.x_bf16 = (x_dtype == BSQ_BF16);
    a.idx = idx;
    a.n = n;
    a.n_total = n_total;
    a.err = err;
    a.d = cfg.d;
    a.b = cfg.b;
    a.h = cfg.hidden;
    a.theta = theta;
    a.lambda_c = hp.lambda_c;
    a.lambda_e = hp.lambda_e;
    a.gamma = hp.gamma;
    a.tau = hp.tau;
    a.cscale = float(1.0 / __builtin_sqrt(double(cfg.b)));
    a.nblk = (n + TB - 1) / TB;
    a.P = train_param_count(cfg);
    a.R = train_record_floats(cfg);
    char *w = static_cast<char *>(ws);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char *p = w + off;
        off += align256(bytes);
        return p;
    };
    a.s_part = reinterpret_cast<float *>(take(size_t(a.nblk) * cfg.b * 4));
    a.h_part = reinterpret_cast<float *>(take(size_t(a.nblk) * 4));
    a.sbar = reinterpret_cast<float *>(take(64));
    a.bar_ent = reinterpret_cast<float *>(take(4));
    a.l_part = reinterpret_cast<float *>(take(size_t(a.nblk) * 8));
    a.rec = reinterpret_cast<float *>(take(size_t(n) * a.R * 4));
    a.g_part = reinterpret_cast<float *>(take(size_t(PG) * a.P * 4));
    a.grad = grad;
    a.loss = loss;
    if (cfg.d == 8) return (cfg.b == 8) ? launch_train_t<8, 8>(a, st) : launch_train_t<8, 16>(a, st);
    return (cfg.b == 8) ? launch_train_t<16, 8>(a, st) : launch_train_t<16, 16>(a, st);
}

hipError_t launch_train_adam(const bsq_config &cfg, const bsq_train_hparams &hp, int step, float *theta,
                             const float *grad, float *m, float *v, hipStream_t st)
{
    AdamArgs a{};
    a.theta = theta;
    a.m = m;
    a.v = v;
    a.grad = grad;
    a.P = train_param_count(cfg);
    a.lr = hp.lr;
    a.beta1 = hp.beta1;
    a.beta2 = hp.beta2;
    a.eps = hp.eps;
    a.bc1 = float(1.0 - __builtin_pow(double(hp.beta1), double(step)));
    a.bc2 = float(1.0 - __builtin_pow(double(hp.beta2), double(step)));
    hipLaunchKernelGGL(train_adam_kernel, dim3(unsigned((a.P + TB - 1) / TB)), dim3(TB), 0, st, a);
    return hipGetLastError();
}

}  // namespace bsq
