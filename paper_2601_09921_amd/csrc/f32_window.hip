// fp32 decoder for small windows: one workgroup runs one window through every round,
// layer and the readout with its whole state in LDS (Algorithm 1, inference branch, or the
// recurrent branch's readout after each of the last rounds; App. A model). Used for the fp32 configurations (d_model <= 64, about d <= 5), where a
// window is a few kilobytes and the batch is small, so one launch per decode is the point.
//
// All matrix products are fp32 FMA loops with the model width as a compile-time constant,
// unrolled with four independent partial sums so the weight loads overlap. Every output
// element is produced by one thread in a fixed order, so results do not depend on the batch.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int THREADS = 512;

struct LayerPtrs {
    const float *Wq, *bq, *Wk, *bk, *Wv, *bv, *Wo, *bo, *g1, *be1, *W1, *b1, *W2, *b2, *g2, *be2;
};

__device__ const float* layer_ptrs(const float* w, int D, int F, int l, LayerPtrs& L) {
    const size_t per = (size_t)4 * D * D + 4 * D + 2 * D + (size_t)D * F + F + (size_t)F * D + 3 * D;
    const float* q = w + 2 * D + per * l;
    L.Wq = q; q += D * D; L.bq = q; q += D;
    L.Wk = q; q += D * D; L.bk = q; q += D;
    L.Wv = q; q += D * D; L.bv = q; q += D;
    L.Wo = q; q += D * D; L.bo = q; q += D;
    L.g1 = q; q += D; L.be1 = q; q += D;
    L.W1 = q; q += (size_t)D * F; L.b1 = q; q += F;
    L.W2 = q; q += (size_t)F * D; L.b2 = q; q += D;
    L.g2 = q; q += D; L.be2 = q; q += D;
    return q;
}

// sum_k in[k] W[k*O + o] for a compile-time K, four interleaved partial sums
template <int K>
PWD_DEV float dot_col(const float* in, const float* __restrict__ W, int O, int o) {
    float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll 8
    for (int k = 0; k < K; k += 4) {
        a0 = fmaf(in[k + 0], W[(size_t)(k + 0) * O + o], a0);
        a1 = fmaf(in[k + 1], W[(size_t)(k + 1) * O + o], a1);
        a2 = fmaf(in[k + 2], W[(size_t)(k + 2) * O + o], a2);
        a3 = fmaf(in[k + 3], W[(size_t)(k + 3) * O + o], a3);
    }
    return (a0 + a1) + (a2 + a3);
}

// out[n][o] = bias[o] + sum_k in[n][k] W[k][o]  (+ res[n][o]); optional ReLU before res
template <int K, int O>
PWD_DEV void linear(const float* in, int N, const float* __restrict__ W, const float* __restrict__ bias,
                    float* out, const float* res, bool relu) {
    for (int idx = threadIdx.x; idx < N * O; idx += THREADS) {
        const int n = idx / O, o = idx % O;
        float acc = bias[o] + dot_col<K>(in + n * K, W, O, o);
        if (relu) acc = fmaxf(acc, 0.f);
        if (res) acc += res[idx];
        out[idx] = acc;
    }
}

// x[n][:] = LayerNorm(x[n][:]) for each token (one thread per token, two passes)
template <int D>
PWD_DEV void layer_norm_rows(float* x, int N, const float* g, const float* b, float eps) {
    for (int n = threadIdx.x; n < N; n += THREADS) {
        float* r = x + n * D;
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < D; ++k) s += r[k];
        const float mean = s / D;
        float v = 0.f;
#pragma unroll
        for (int k = 0; k < D; ++k) v += (r[k] - mean) * (r[k] - mean);
        const float rstd = rsqrtf(v / D + eps);
#pragma unroll
        for (int k = 0; k < D; ++k) r[k] = (r[k] - mean) * rstd * g[k] + b[k];
    }
}

template <int D, int MR>
__global__ __launch_bounds__(THREADS) void f32_window_kernel(F32Params p) {
    constexpr int F = MR * D;   // feed-forward width
    const int win = blockIdx.x;
    const int N = p.ntok, H = p.H, dh = D / H, d = p.in.d;
    extern __shared__ __align__(16) float sm[];
    float* X = sm;                 // [N][D] state / residual stream
    float* Z = X + N * D;          // [N][D] scratch
    float* Q = Z + N * D;          // [N][D]
    float* K = Q + N * D;          // [N][D]
    float* V = K + N * D;          // [N][D]
    float* A = V + N * D;          // [N][D] attention output (heads concatenated)
    float* Hd = A + N * D;         // [N][F] feed-forward hidden
    float* S = Hd + N * F;         // [H][N][N] scores / probabilities
    __shared__ uint32_t ev[32];    // event words of one round (at most 1024 stabilizers)
    __shared__ float red[THREADS];

    const int type = p.in.types[win];
    const uint32_t* meas = p.in.meas + (int64_t)win * (p.in.W + 1) * p.in.words;
    const float* we = p.w;
    const float scale = rsqrtf((float)dh);

    // readout (App. A.3) of the current state into output slot k: 2x2 valid convolution +
    // ReLU, mean over columns, linear; one fixed-order reduction over the workgroup
    auto readout = [&](int k) {
        LayerPtrs L;
        const float* Wc = layer_ptrs(p.w, D, F, p.L - 1, L);
        const float* bc = Wc + 4 * (size_t)D * D;
        const float* wo = bc + D;
        const float bo = wo[(size_t)d * D];
        const float* beta = wo + (size_t)d * D + 1;
        const int gw = d + 1;
        float part = 0.f;
        for (int idx = threadIdx.x; idx < d * D; idx += THREADS) {
            const int i = idx / D, o = idx % D;
            float pool = 0.f;
            for (int j = 0; j < d; ++j) {
                float acc = bc[o];
                for (int a = 0; a < 2; ++a)
                    for (int b = 0; b < 2; ++b) {
                        const int tok = p.cell_token[(i + a) * gw + (j + b)];
                        if (tok < 0) continue;
                        acc += dot_col<D>(X + tok * D, Wc + (size_t)(a * 2 + b) * D * D, D, o);
                    }
                pool += fmaxf(acc, 0.f);
            }
            part = fmaf(wo[idx], pool / (float)d, part);
        }
        red[threadIdx.x] = part;
        __syncthreads();
        for (int n = THREADS / 2; n > 0; n >>= 1) {
            if ((int)threadIdx.x < n) red[threadIdx.x] += red[threadIdx.x + n];
            __syncthreads();
        }
        if (threadIdx.x == 0) {
            const int64_t o = (int64_t)win * p.readouts + k;
            if (type > WIN_FINAL) {
                p.logits[o] = __builtin_nanf("");
                p.bits[o] = 0;
                atomicOr(p.err, 1);
            } else {
                const float logit = red[0] + bo + beta[type];
                p.logits[o] = logit;
                p.bits[o] = logit > 0.f ? 1 : 0;
            }
        }
        __syncthreads();   // red is reused by the next readout
    };

    for (int t = 0; t < p.in.W; ++t) {
        for (int wd = threadIdx.x; wd < p.in.words; wd += THREADS)
            ev[wd] = type > WIN_FINAL ? 0u : event_word(meas, p.in.words, t, wd, type, p.in.b_left, d);
        __syncthreads();
        // embedding + fold: X = kappa (E w_e + b_e + PE + X), X = 0 before round 0; with the
        // embedder's residual block, plus its output looked up by the events of the five cells
        // around the token's cell and the cell's position class
        auto ev_bit = [&](int st) { return st >= 0 ? (ev[st >> 5] >> (st & 31)) & 1u : 0u; };
        for (int idx = threadIdx.x; idx < N * D; idx += THREADS) {
            const int n = idx / D, k = idx % D;
            const int st = p.tok_stab ? p.tok_stab[n] : n;   // the token's stabilizer, or -1
            const float e = (float)ev_bit(st);
            float s = fmaf(e, we[k], p.S0[idx]);
            if (p.emb_tab) {
                const int* nb = p.emb_nb + n * 8;
                uint32_t pat = 0u;
                for (int j = 0; j < 5; ++j) pat |= ev_bit(nb[j]) << j;
                s += p.emb_tab[(size_t)(nb[5] * 32 + (int)pat) * D + k];
            }
            X[idx] = p.kappa * (s + (t > 0 ? X[idx] : 0.f));
        }
        __syncthreads();
        for (int l = 0; l < p.L; ++l) {
            LayerPtrs L;
            layer_ptrs(p.w, D, F, l, L);
            linear<D, D>(X, N, L.Wq, L.bq, Q, nullptr, false);
            linear<D, D>(X, N, L.Wk, L.bk, K, nullptr, false);
            linear<D, D>(X, N, L.Wv, L.bv, V, nullptr, false);
            __syncthreads();
            for (int idx = threadIdx.x; idx < H * N * N; idx += THREADS) {
                const int h = idx / (N * N), q = (idx / N) % N, k = idx % N;
                float acc = 0.f;
                for (int e = 0; e < dh; ++e) acc = fmaf(Q[q * D + h * dh + e], K[k * D + h * dh + e], acc);
                S[idx] = acc * scale;
            }
            __syncthreads();
            for (int row = threadIdx.x; row < H * N; row += THREADS) {
                float* r = S + row * N;
                float mx = r[0];
                for (int k = 1; k < N; ++k) mx = fmaxf(mx, r[k]);
                float sum = 0.f;
                for (int k = 0; k < N; ++k) {
                    r[k] = expf(r[k] - mx);
                    sum += r[k];
                }
                const float inv = 1.f / sum;
                for (int k = 0; k < N; ++k) r[k] *= inv;
            }
            __syncthreads();
            for (int idx = threadIdx.x; idx < N * D; idx += THREADS) {
                const int q = idx / D, c = idx % D, h = c / dh;
                float acc = 0.f;
                for (int k = 0; k < N; ++k) acc = fmaf(S[(h * N + q) * N + k], V[k * D + c], acc);
                A[idx] = acc;
            }
            __syncthreads();
            linear<D, D>(A, N, L.Wo, L.bo, Z, X, false);      // Z = X + A Wo + bo
            __syncthreads();
            layer_norm_rows<D>(Z, N, L.g1, L.be1, p.eps);
            __syncthreads();
            if (p.conv_w) {
                // dilated convolutions on the grid (token = cell): three residual units
                // Z += ReLU(b_j + sum_{a,e} Z[cell + dil_j (a-1, e-1)] Wd_j[a][e]); A is free
                const float* cw = p.conv_w + (size_t)l * (27 * (size_t)D * D + 3 * D);
                const int side = d + 1;
                for (int j = 0; j < 3; ++j) {
                    const float* Wj = cw + (size_t)j * 9 * D * D;
                    const float* bj = cw + 27 * (size_t)D * D + j * D;
                    for (int idx = threadIdx.x; idx < N * D; idx += THREADS) {
                        const int n = idx / D, o = idx % D, r = n / side, c = n % side;
                        float acc = bj[o];
                        for (int tap = 0; tap < 9; ++tap) {
                            const int rr = r + p.dil[j] * (tap / 3 - 1), cc = c + p.dil[j] * (tap % 3 - 1);
                            if (rr < 0 || rr >= side || cc < 0 || cc >= side) continue;
                            acc += dot_col<D>(Z + (rr * side + cc) * D, Wj + (size_t)tap * D * D, D, o);
                        }
                        A[idx] = fmaxf(acc, 0.f);
                    }
                    __syncthreads();
                    for (int idx = threadIdx.x; idx < N * D; idx += THREADS) Z[idx] += A[idx];
                    __syncthreads();
                }
            }
            linear<D, F>(Z, N, L.W1, L.b1, Hd, nullptr, true);
            __syncthreads();
            linear<F, D>(Hd, N, L.W2, L.b2, X, Z, false);     // X = Z + FF(Z)
            __syncthreads();
            layer_norm_rows<D>(X, N, L.g2, L.be2, p.eps);
            __syncthreads();
        }
        if (t >= p.in.W - p.readouts) readout(t - (p.in.W - p.readouts));
    }
}

template <int D, int MR>
hipError_t launch_dm(const F32Params& p, hipStream_t s) {
    const size_t smem = f32_window_smem_bytes(p.ntok, p.D, p.H, p.F);
    hipError_t e = hipFuncSetAttribute((const void*)f32_window_kernel<D, MR>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    f32_window_kernel<D, MR><<<dim3((unsigned)p.in.nwin), dim3(THREADS), smem, s>>>(p);
    return hipGetLastError();
}

template <int D>
hipError_t launch_d(const F32Params& p, hipStream_t s) {
    if (p.F == 4 * D) return launch_dm<D, 4>(p, s);
    if (p.F == 5 * D) return launch_dm<D, 5>(p, s);
    return hipErrorInvalidValue;
}

}  // namespace

size_t f32_window_smem_bytes(int N, int D, int H, int F) {
    return ((size_t)6 * N * D + (size_t)N * F + (size_t)H * N * N) * sizeof(float);
}

hipError_t launch_f32_window(const F32Params& p, hipStream_t s) {
    if (p.in.nwin <= 0) return hipSuccess;
    switch (p.D) {
        case 16: return launch_d<16>(p, s);
        case 32: return launch_d<32>(p, s);
        case 64: return launch_d<64>(p, s);
        default: return hipErrorInvalidValue;
    }
}
