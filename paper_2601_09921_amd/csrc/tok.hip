// Token-local stages of one Syndrome Transformer step, fused per token (bf16 MFMA path).
//
// One launch runs, for 32 tokens per wavefront, any of:
//   POST : out-projection of the attention output, residual, LayerNorm 1, feed-forward
//          D -> F -> D with ReLU, residual, LayerNorm 2 (App. A.2 Syndrome Transformer;
//          post-norm residual blocks).
//   EMBED: the stabilizer embedding of round t and the recurrent fold
//          X = kappa * (E_t w_e + b_e + PE + X) (App. A.1 embedder and positional
//          encoding; App. A.2 fold equation; Algorithm 1, D_0 = 0 at t = 0).
//   QKV  : the Q, K, V projections of the following layer.
// The residual stream stays fp32 in registers; only GEMM operands are rounded to bf16.
// GEMMs are transposed (Out^T = W^T In^T) so tokens lie along MFMA columns: LayerNorm
// reduces over the four lanes that share a token, and each accumulator becomes the next
// GEMM's B operand in registers.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int TB = 2;        // 16-token blocks per wavefront
constexpr int WAVES = 4;     // wavefronts per workgroup
constexpr int CH = 64;       // feed-forward hidden units per chunk

PWD_DEV bf16x8 ldfrag(const uint16_t* __restrict__ base, int64_t frag, int lane) {
    const u16x8 v = *reinterpret_cast<const u16x8*>(base + (frag * 64 + lane) * 8);
    return __builtin_bit_cast(bf16x8, v);
}

PWD_DEV void stfrag(uint16_t* __restrict__ base, int64_t frag, int lane, bf16x8 v) {
    *reinterpret_cast<u16x8*>(base + (frag * 64 + lane) * 8) = __builtin_bit_cast(u16x8, v);
}

PWD_DEV f32x4 ld4(const float* __restrict__ p) { return *reinterpret_cast<const f32x4*>(p); }

PWD_DEV f32x4 relu4(f32x4 v) {
    f32x4 r;
    #pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = v[i] > 0.f ? v[i] : 0.f;
    return r;
}

// LayerNorm over the D features of each token (biased variance, two passes).
template <int RT>
PWD_DEV void layer_norm(f32x4 (&x)[RT][TB], const float* __restrict__ gamma,
                        const float* __restrict__ beta, float eps, int g) {
    constexpr float inv_d = 1.0f / (RT * 16);
    #pragma unroll
    for (int b = 0; b < TB; ++b) {
        float s = 0.f;
        #pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            s += (x[rt][b][0] + x[rt][b][1]) + (x[rt][b][2] + x[rt][b][3]);
        s += __shfl_xor(s, 16);
        s += __shfl_xor(s, 32);
        const float mean = s * inv_d;
        float v = 0.f;
        #pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            #pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float c = x[rt][b][i] - mean;
                v += c * c;
            }
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        const float rstd = rsqrtf(v * inv_d + eps);
        #pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 gm = ld4(gamma + rt * 16 + 4 * g);
            const f32x4 bt = ld4(beta + rt * 16 + 4 * g);
            #pragma unroll
            for (int i = 0; i < 4; ++i) x[rt][b][i] = (x[rt][b][i] - mean) * rstd * gm[i] + bt[i];
        }
    }
}

template <int D, int FLAGS>
__global__ __launch_bounds__(WAVES * 64) void tok_kernel(TokParams p) {
    constexpr int RT = D / 16;   // 16-row C tiles per activation
    constexpr int KS = D / 32;   // 32-deep k-steps per activation
    const int lane = threadIdx.x & 63;
    const int g = lane >> 4;
    const int col = lane & 15;
    const int64_t tb0 = ((int64_t)blockIdx.x * WAVES + (threadIdx.x >> 6)) * TB;

    f32x4 x[RT][TB];

    if constexpr ((FLAGS & TOK_POST) != 0) {
        // ---- out-projection + residual + LayerNorm 1; accumulators start at X + b_o
        {
            bf16x8 y[KS][TB];
            #pragma unroll
            for (int b = 0; b < TB; ++b)
                #pragma unroll
                for (int ks = 0; ks < KS; ++ks) y[ks][b] = ldfrag(p.Y, (tb0 + b) * KS + ks, lane);
            #pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const f32x4 bias = ld4(p.bo + rt * 16 + 4 * g);
                #pragma unroll
                for (int b = 0; b < TB; ++b)
                    x[rt][b] = ld4(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4) + bias;
            }
            #pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                #pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 a = ldfrag(p.Wo, rt * KS + ks, lane);
                    #pragma unroll
                    for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, y[ks][b], x[rt][b]);
                }
        }
        layer_norm<RT>(x, p.g1, p.be1, p.eps, g);

        // ---- feed-forward, hidden units in chunks of CH; accumulators start at X + b_2
        bf16x8 xb[KS][TB];
        #pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            #pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        #pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 bias = ld4(p.b2 + rt * 16 + 4 * g);
            #pragma unroll
            for (int b = 0; b < TB; ++b) x[rt][b] += bias;
        }
        constexpr int F = 4 * D;
        constexpr int FKS = F / 32;
        for (int c = 0; c < F / CH; ++c) {
            f32x4 h[CH / 16][TB];
            #pragma unroll
            for (int rh = 0; rh < CH / 16; ++rh) {
                const f32x4 bias = ld4(p.b1 + c * CH + rh * 16 + 4 * g);
                #pragma unroll
                for (int b = 0; b < TB; ++b) h[rh][b] = bias;
            }
            #pragma unroll
            for (int rh = 0; rh < CH / 16; ++rh)
                #pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 a = ldfrag(p.W1, (c * (CH / 16) + rh) * KS + ks, lane);
                    #pragma unroll
                    for (int b = 0; b < TB; ++b) h[rh][b] = mfma16x16x32(a, xb[ks][b], h[rh][b]);
                }
            bf16x8 hb[CH / 32][TB];
            #pragma unroll
            for (int kh = 0; kh < CH / 32; ++kh)
                #pragma unroll
                for (int b = 0; b < TB; ++b)
                    hb[kh][b] = pack_b(relu4(h[2 * kh][b]), relu4(h[2 * kh + 1][b]));
            #pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                #pragma unroll
                for (int kh = 0; kh < CH / 32; ++kh) {
                    const bf16x8 a = ldfrag(p.W2, rt * FKS + c * (CH / 32) + kh, lane);
                    #pragma unroll
                    for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, hb[kh][b], x[rt][b]);
                }
        }
        layer_norm<RT>(x, p.g2, p.be2, p.eps, g);
    }

    if constexpr ((FLAGS & TOK_EMBED) != 0) {
        // ---- embedding of round t folded into the state: X = kappa (S_t + X)
        #pragma unroll
        for (int b = 0; b < TB; ++b) {
            const int64_t tb = tb0 + b;
            const int64_t w = tb / p.nbw;
            const int blk = (int)(tb - w * p.nbw);
            const int s = blk * 16 + col;
            float e = 0.f;
            if (w < p.in.nwin && s < p.in.N) {
                const uint32_t* m = p.in.meas + w * (int64_t)(p.in.W + 1) * p.in.words;
                const uint32_t word = event_word(m, p.in.words, p.t, s >> 5, p.in.types[w],
                                                 p.in.b_left, p.in.d);
                e = (float)((word >> (s & 31)) & 1u);
            }
            #pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const f32x4 s0 = ld4(p.S0 + (((int64_t)blk * RT + rt) * 64 + lane) * 4);
                const f32x4 we = ld4(p.we + rt * 16 + 4 * g);
                const bool real = s < p.in.N;
                #pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float emb = real ? e * we[i] + s0[i] : 0.f;
                    const float prev = (FLAGS & TOK_POST) ? x[rt][b][i] : 0.f;
                    x[rt][b][i] = p.kappa * (emb + prev);
                }
            }
        }
    }

    #pragma unroll
    for (int b = 0; b < TB; ++b)
        #pragma unroll
        for (int rt = 0; rt < RT; ++rt)
            *reinterpret_cast<f32x4*>(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4) = x[rt][b];

    if constexpr ((FLAGS & TOK_QKV) != 0) {
        bf16x8 xb[KS][TB];
        #pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            #pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        // 3D output features in groups of 32 (= one B fragment of Q, K or V)
        #pragma unroll
        for (int og = 0; og < 3 * KS; ++og) {
            f32x4 q0[TB], q1[TB];
            const f32x4 bias0 = ld4(p.bqkv + og * 32 + 4 * g);
            const f32x4 bias1 = ld4(p.bqkv + og * 32 + 16 + 4 * g);
            #pragma unroll
            for (int b = 0; b < TB; ++b) {
                q0[b] = bias0;
                q1[b] = bias1;
            }
            #pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 a0 = ldfrag(p.Wqkv, (2 * og) * KS + ks, lane);
                const bf16x8 a1 = ldfrag(p.Wqkv, (2 * og + 1) * KS + ks, lane);
                #pragma unroll
                for (int b = 0; b < TB; ++b) {
                    q0[b] = mfma16x16x32(a0, xb[ks][b], q0[b]);
                    q1[b] = mfma16x16x32(a1, xb[ks][b], q1[b]);
                }
            }
            #pragma unroll
            for (int b = 0; b < TB; ++b) stfrag(p.QKV, (tb0 + b) * (3 * KS) + og, lane, pack_b(q0[b], q1[b]));
        }
    }
}

template <int D>
hipError_t launch_tok_d(int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    const int64_t per_wg = (int64_t)WAVES * TB;
    const dim3 grid((unsigned)((n_tb + per_wg - 1) / per_wg)), block(WAVES * 64);
    switch (flags) {
        case TOK_EMBED | TOK_QKV: tok_kernel<D, TOK_EMBED | TOK_QKV><<<grid, block, 0, s>>>(p); break;
        case TOK_POST | TOK_QKV: tok_kernel<D, TOK_POST | TOK_QKV><<<grid, block, 0, s>>>(p); break;
        case TOK_POST | TOK_EMBED | TOK_QKV:
            tok_kernel<D, TOK_POST | TOK_EMBED | TOK_QKV><<<grid, block, 0, s>>>(p); break;
        case TOK_POST: tok_kernel<D, TOK_POST><<<grid, block, 0, s>>>(p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

// Token blocks are processed in groups of WAVES*TB; every buffer indexed here must be
// allocated for n_tb rounded up to that multiple.
int64_t tok_block_granule() { return (int64_t)WAVES * TB; }

hipError_t launch_tok(int D, int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    if (n_tb <= 0) return hipSuccess;
    if (D == 256) return launch_tok_d<256>(flags, p, n_tb, s);
    if (D == 128) return launch_tok_d<128>(flags, p, n_tb, s);
    return hipErrorInvalidValue;
}
