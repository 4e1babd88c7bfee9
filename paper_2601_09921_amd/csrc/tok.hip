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
//
// Weights reach the MFMAs through LDS: the host lays every weight fragment out in the exact
// order the kernel consumes them (a "weight stream"), and the workgroup pulls the stream
// through a double-buffered LDS ring in 32 KB chunks with direct global->LDS loads, one
// chunk ahead of the MFMAs. Every fragment read from LDS feeds 2-3 MFMAs of each wavefront
// (one per 16-token block the wavefront owns).
#include "common.h"
#include "kernels.h"

#include <type_traits>

namespace {

constexpr int WAVES = 4;        // wavefronts per workgroup
constexpr int MAX_CHUNK = 64;   // weight fragments (1 KB each) per LDS chunk, at most
constexpr int FRAG = 512;       // bf16 values per fragment

// 16-token blocks per wavefront: three where the registers allow it (more tokens per
// workgroup share each streamed weight chunk), else two.
template <int D, int FLAGS>
constexpr int tok_tb() { return (D == 256 && (FLAGS & TOK_EMBED) == 0) ? 3 : 2; }

template <int D, int TB>
struct Shape {
    static constexpr int CHUNK = (D == 256 && TB == 2) ? 64 : 32;  // weight fragments per LDS chunk
    static constexpr int RT = D / 16;                 // 16-row C tiles of a D-vector
    static constexpr int KS = D / 32;                 // 32-deep k-steps of a D-vector
    static constexpr int F = 4 * D;
    static constexpr int CH = 8192 / D;               // hidden units per feed-forward chunk
    static constexpr int NMLP = F / CH;               // feed-forward sub-chunks (32 fragments each)
    static constexpr int MLP_PER = CHUNK / 32;        // feed-forward sub-chunks per LDS chunk
    static constexpr int MLP_CHUNKS = NMLP / MLP_PER;
    static constexpr int WO_CHUNKS = RT * KS / CHUNK;
    static constexpr int QKV_CHUNKS = (3 * D / 16) * KS / CHUNK;
    static constexpr int OG_PER_CHUNK = CHUNK / (2 * KS);
    static constexpr int POST_CHUNKS = WO_CHUNKS + MLP_CHUNKS;
    static_assert((CH / 16) * KS + RT * (CH / 32) == 32, "32 fragments per feed-forward sub-chunk");
    static_assert(NMLP % MLP_PER == 0 && CHUNK <= MAX_CHUNK, "whole feed-forward chunks");
    static_assert(RT * KS % CHUNK == 0 && (3 * D / 16) * KS % CHUNK == 0, "whole chunks");
};

PWD_DEV bf16x8 ldfrag(const uint16_t* __restrict__ base, int64_t frag, int lane) {
    const u16x8 v = *reinterpret_cast<const u16x8*>(base + (frag * 64 + lane) * 8);
    return __builtin_bit_cast(bf16x8, v);
}

PWD_DEV bf16x8 lds_frag(const uint16_t* buf, int j, int lane) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(buf + j * FRAG + lane * 8));
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

// Scheduling shape of a chunk: LA LDS reads first, then (MPR MFMAs, 1 LDS read) pairs, then
// the last MFMAs, so LA fragment reads stay in flight ahead of the matrix core.
template <int NREAD, int MPR, int LA>
PWD_DEV void sched_pipeline() {
    __builtin_amdgcn_sched_group_barrier(0x100, LA, 0);
#pragma unroll
    for (int k = 0; k < NREAD - LA; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, MPR, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, MPR * LA, 0);
}

// The two LDS buffers of the weight stream. They are separate objects so the compiler can
// tell that the direct-to-LDS prefetch into one never aliases reads of the other.
template <int PAR, int CHUNK>
PWD_DEV uint16_t* wbuf() {
    static_assert(CHUNK <= MAX_CHUNK, "chunk size");
    __shared__ __align__(16) uint16_t buf[CHUNK * FRAG];   // one object per (buffer, size)
    return buf;
}

// The weight stream of one launch: `post` chunks first, then `qkv` chunks, pulled through
// the two LDS buffers (chunk i lives in buffer i % 2). begin<i % 2>(i) makes chunk i visible
// to every wavefront and starts the load of chunk i+1 into the other buffer.
template <int CHUNK>
struct WeightPipe {
    const uint16_t* post;
    const uint16_t* qkv;
    int n_post, total;
    int lane, wave;

    template <int PAR>
    __device__ void issue(int i) const {
        const uint16_t* src = i < n_post ? post + (size_t)i * CHUNK * FRAG
                                         : qkv + (size_t)(i - n_post) * CHUNK * FRAG;
        uint16_t* dst = wbuf<PAR, CHUNK>();
#pragma unroll
        for (int j = 0; j < CHUNK / WAVES; ++j) {
            const int f = wave * (CHUNK / WAVES) + j;
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(src + (f * 64 + lane) * 8),
                (__attribute__((address_space(3))) void*)(dst + f * FRAG), 16, 0, 0);
        }
    }
    // Chunk i is visible to every wavefront after sync(i); prefetch(i) then starts chunk
    // i+1. LDS reads of other tables belong between the two: no prefetch is in flight then,
    // so the compiler has nothing to wait for.
    template <int PAR>
    __device__ const uint16_t* sync(int) const {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this wave's part of chunk i landed
        __syncthreads();                                   // ... and everyone's; buffer i-1 is free
        return wbuf<PAR, CHUNK>();
    }
    template <int PAR>
    __device__ void prefetch(int i) const {
        if (i + 1 < total) issue<1 - PAR>(i + 1);
        __builtin_amdgcn_sched_barrier(0);                 // keep the prefetch ahead of the MFMAs
    }
    template <int PAR>
    __device__ const uint16_t* begin(int i) const {
        const uint16_t* b = sync<PAR>(i);
        prefetch<PAR>(i);
        return b;
    }
};

// LayerNorm over the D features of each token (biased variance, two passes); gamma and
// beta are in LDS.
template <int RT, int TB>
PWD_DEV void layer_norm(f32x4 (&x)[RT][TB], const float* gamma, const float* beta, float eps, int g) {
    constexpr float inv_d = 1.0f / (RT * 16);
#pragma unroll
    for (int b = 0; b < TB; ++b) {
        float s = 0.f;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) s += (x[rt][b][0] + x[rt][b][1]) + (x[rt][b][2] + x[rt][b][3]);
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

// Per-launch vectors staged in LDS once: [bo g1 be1 b2 g2 be2 | b1 (F) | bqkv (3D)].
template <int D>
struct Vecs {
    static constexpr int BO = 0, G1 = D, BE1 = 2 * D, B2 = 3 * D, G2 = 4 * D, BE2 = 5 * D;
    static constexpr int B1 = 6 * D, BQKV = 10 * D, SIZE = 13 * D;
};

template <int D, int FLAGS>
__global__ __launch_bounds__(WAVES * 64, 1) void tok_kernel(TokParams p) {
    constexpr int TB = tok_tb<D, FLAGS>();
    using S = Shape<D, TB>;
    using V = Vecs<D>;
    constexpr int RT = S::RT, KS = S::KS, CH = S::CH;
    constexpr bool POST = (FLAGS & TOK_POST) != 0, QKV = (FLAGS & TOK_QKV) != 0;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 4;
    const int col = lane & 15;
    const int64_t tb0 = ((int64_t)blockIdx.x * WAVES + wave) * TB;

    constexpr int CHUNK = S::CHUNK;
    WeightPipe<CHUNK> pipe;
    pipe.post = p.post_stream;
    pipe.qkv = p.qkv_stream;
    pipe.n_post = POST ? S::POST_CHUNKS : 0;
    pipe.total = pipe.n_post + (QKV ? S::QKV_CHUNKS : 0);
    pipe.lane = lane;
    pipe.wave = wave;
    pipe.template issue<0>(0);

    __shared__ __align__(16) float vec[V::SIZE];
    if (POST) {
        const float* src[7] = {p.bo, p.g1, p.be1, p.b2, p.g2, p.be2, p.b1};
        for (int k = 0; k < 6; ++k)
            for (int i = threadIdx.x; i < D; i += WAVES * 64) vec[k * D + i] = src[k][i];
        for (int i = threadIdx.x; i < 4 * D; i += WAVES * 64) vec[V::B1 + i] = src[6][i];
    }
    if (QKV)
        for (int i = threadIdx.x; i < 3 * D; i += WAVES * 64) vec[V::BQKV + i] = p.bqkv[i];
    // (the first pipe.begin's barrier publishes vec)

    f32x4 x[RT][TB];

    if constexpr (POST) {
        // ---- out-projection + residual + LayerNorm 1; accumulators start at X (+ b_o below)
        {
            bf16x8 y[KS][TB];
#pragma unroll
            for (int b = 0; b < TB; ++b)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) y[ks][b] = ldfrag(p.Y, (tb0 + b) * KS + ks, lane);
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int b = 0; b < TB; ++b) x[rt][b] = ld4(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4);
            auto wo_chunk = [&](const uint16_t* buf, int c) {
#pragma unroll
                for (int j = 0; j < CHUNK; ++j) {
                    const int fr = c * CHUNK + j, rt = fr / KS, ks = fr % KS;
                    const bf16x8 a = lds_frag(buf, j, lane);
#pragma unroll
                    for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, y[ks][b], x[rt][b]);
                }
                sched_pipeline<CHUNK, TB, 4>();
            };
            static_assert(S::WO_CHUNKS == 1 || S::WO_CHUNKS % 2 == 0, "Wo chunks");
            if constexpr (S::WO_CHUNKS == 1) {
                wo_chunk(pipe.template begin<0>(0), 0);
            } else {
#pragma unroll
                for (int c = 0; c < S::WO_CHUNKS; c += 2) {
                    wo_chunk(pipe.template begin<0>(c), c);
                    wo_chunk(pipe.template begin<1>(c + 1), c + 1);
                }
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 bias = ld4(vec + V::BO + rt * 16 + 4 * g);
#pragma unroll
            for (int b = 0; b < TB; ++b) x[rt][b] += bias;
        }
        layer_norm<RT, TB>(x, vec + V::G1, vec + V::BE1, p.eps, g);

        // ---- feed-forward, hidden units in chunks of CH; accumulators start at X + b_2
        bf16x8 xb[KS][TB];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 bias = ld4(vec + V::B2 + rt * 16 + 4 * g);
#pragma unroll
            for (int b = 0; b < TB; ++b) x[rt][b] += bias;
        }
        auto mlp_sub = [&](const uint16_t* buf, const f32x4 (&bias)[CH / 16]) {
            f32x4 h[CH / 16][TB];
#pragma unroll
            for (int rh = 0; rh < CH / 16; ++rh)
#pragma unroll
                for (int b = 0; b < TB; ++b) h[rh][b] = bias[rh];
#pragma unroll
            for (int rh = 0; rh < CH / 16; ++rh)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 a = lds_frag(buf, rh * KS + ks, lane);
#pragma unroll
                    for (int b = 0; b < TB; ++b) h[rh][b] = mfma16x16x32(a, xb[ks][b], h[rh][b]);
                }
            bf16x8 hb[CH / 32][TB];
#pragma unroll
            for (int kh = 0; kh < CH / 32; ++kh)
#pragma unroll
                for (int b = 0; b < TB; ++b) hb[kh][b] = pack_b(relu4(h[2 * kh][b]), relu4(h[2 * kh + 1][b]));
            const uint16_t* w2 = buf + (CH / 16) * KS * FRAG;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int kh = 0; kh < CH / 32; ++kh) {
                    const bf16x8 a = lds_frag(w2, rt * (CH / 32) + kh, lane);
#pragma unroll
                    for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, hb[kh][b], x[rt][b]);
                }
        };
        constexpr int MP = S::MLP_PER;
        auto mlp_chunk = [&](auto par, int c) {
            constexpr int PAR = decltype(par)::value;
            const int ci = S::WO_CHUNKS + c;
            const uint16_t* buf = pipe.template sync<PAR>(ci);
            f32x4 bias[MP][CH / 16];
#pragma unroll
            for (int u = 0; u < MP; ++u)
#pragma unroll
                for (int rh = 0; rh < CH / 16; ++rh)
                    bias[u][rh] = ld4(vec + V::B1 + (c * MP + u) * CH + rh * 16 + 4 * g);
            pipe.template prefetch<PAR>(ci);
#pragma unroll
            for (int u = 0; u < MP; ++u) mlp_sub(buf + u * 32 * FRAG, bias[u]);
            sched_pipeline<MP * (CH / 16 + 32), TB, 6>();
        };
        static_assert(S::MLP_CHUNKS % 2 == 0, "feed-forward chunks come in pairs");
        constexpr int P0 = S::WO_CHUNKS & 1;
        for (int c = 0; c < S::MLP_CHUNKS; c += 2) {
            mlp_chunk(std::integral_constant<int, P0>{}, c);
            mlp_chunk(std::integral_constant<int, 1 - P0>{}, c + 1);
        }
        layer_norm<RT, TB>(x, vec + V::G2, vec + V::BE2, p.eps, g);
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
            const bool real = s < p.in.N;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const f32x4 s0 = ld4(p.S0 + (((int64_t)blk * RT + rt) * 64 + lane) * 4);
                const f32x4 we = ld4(p.we + rt * 16 + 4 * g);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float emb = real ? e * we[i] + s0[i] : 0.f;
                    const float prev = POST ? x[rt][b][i] : 0.f;
                    x[rt][b][i] = p.kappa * (emb + prev);
                }
            }
        }
    }

    auto store_x = [&]() {
#pragma unroll
        for (int b = 0; b < TB; ++b)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                *reinterpret_cast<f32x4*>(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4) = x[rt][b];
    };

    store_x();
    if constexpr (QKV) {
        bf16x8 xb[KS][TB];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        // 3D output features in groups of 32 (= one B fragment of Q, K or V)
        constexpr int NP = POST ? S::POST_CHUNKS : 0;
        constexpr int OPC = S::OG_PER_CHUNK;
        auto qkv_chunk = [&](auto par, int qc) {
            constexpr int PAR = decltype(par)::value;
            const uint16_t* buf = pipe.template sync<PAR>(NP + qc);
            f32x4 bias[OPC][2];
#pragma unroll
            for (int o2 = 0; o2 < OPC; ++o2)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh)
                    bias[o2][hh] = ld4(vec + V::BQKV + (qc * OPC + o2) * 32 + hh * 16 + 4 * g);
            pipe.template prefetch<PAR>(NP + qc);
#pragma unroll
            for (int o2 = 0; o2 < OPC; ++o2) {
                const int og = qc * OPC + o2;
                f32x4 q0[TB], q1[TB];
#pragma unroll
                for (int b = 0; b < TB; ++b) {
                    q0[b] = bias[o2][0];
                    q1[b] = bias[o2][1];
                }
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const bf16x8 a0 = lds_frag(buf, (o2 * KS + ks) * 2, lane);
                    const bf16x8 a1 = lds_frag(buf, (o2 * KS + ks) * 2 + 1, lane);
#pragma unroll
                    for (int b = 0; b < TB; ++b) {
                        q0[b] = mfma16x16x32(a0, xb[ks][b], q0[b]);
                        q1[b] = mfma16x16x32(a1, xb[ks][b], q1[b]);
                    }
                }
                const float sc = og < KS ? p.qscale : 1.0f;   // Q: log2(e)/sqrt(dh)
#pragma unroll
                for (int b = 0; b < TB; ++b)
                    stfrag(p.QKV, (tb0 + b) * (3 * KS) + og, lane, pack_b(q0[b] * sc, q1[b] * sc));
            }
            sched_pipeline<CHUNK, TB, 6>();
        };
        constexpr int Q0 = NP & 1;
        int qc = 0;
        for (; qc + 1 < S::QKV_CHUNKS; qc += 2) {
            qkv_chunk(std::integral_constant<int, Q0>{}, qc);
            qkv_chunk(std::integral_constant<int, 1 - Q0>{}, qc + 1);
        }
        if constexpr (S::QKV_CHUNKS % 2 == 1) qkv_chunk(std::integral_constant<int, Q0>{}, qc);
    }
}

template <int D, int FLAGS>
void launch_variant(const TokParams& p, int64_t n_tb, hipStream_t s) {
    const int64_t per_wg = (int64_t)WAVES * tok_tb<D, FLAGS>();
    const dim3 grid((unsigned)((n_tb + per_wg - 1) / per_wg)), block(WAVES * 64);
    tok_kernel<D, FLAGS><<<grid, block, 0, s>>>(p);
}

template <int D>
hipError_t launch_tok_d(int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    switch (flags) {
        case TOK_EMBED | TOK_QKV: launch_variant<D, TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST | TOK_QKV: launch_variant<D, TOK_POST | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST | TOK_EMBED | TOK_QKV: launch_variant<D, TOK_POST | TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST: launch_variant<D, TOK_POST>(p, n_tb, s); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

// Token blocks are processed in groups of WAVES*TB (TB = 2 or 3 by variant); every buffer
// indexed here must be allocated for n_tb rounded up to a multiple of all of them.
int64_t tok_block_granule() { return (int64_t)WAVES * 6; }

// Fragments of the weight streams (see tok_kernel): hidden units per feed-forward chunk.
int tok_mlp_chunk(int D) { return 8192 / D; }

hipError_t launch_tok(int D, int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    if (n_tb <= 0) return hipSuccess;
    if (D == 256) return launch_tok_d<256>(flags, p, n_tb, s);
    if (D == 128) return launch_tok_d<128>(flags, p, n_tb, s);
    return hipErrorInvalidValue;
}
