// The recurrent decoder with each window's state resident on chip for all rounds and layers
// (Algorithm 1: the state D_n is carried from round to round, D_0 = 0; App. A.2 fold and
// Syndrome Transformer layers), bf16 MFMA with fp32 state, accumulation, softmax and LayerNorm.
//
// One wavefront owns one whole window of up to four 16-token blocks (the 48 stabilizers of
// d = 7 are three). Its fp32 state stays in registers through every round and layer, and so
// do the window's Q, K and V: the projections are computed transposed with tokens along MFMA
// columns, so after a bf16 pack their accumulators are exactly the operands attention takes --
// K as the A operand of S^T = K Q'^T, Q' = Q log2(e)/sqrt(dh) as its B operand, and V,
// computed with the activations as the A operand (tokens as rows), as the A operand of
// O^T = V^T P^T; the output O^T packs into the B operand of the out-projection. Attention is
// local to the wavefront. Softmax is shift-invariant, so the scores are exponentiated as they
// are; a head whose row sums or outputs leave the normal fp32 range (possible only for scores
// beyond about +-100 log2 units) is recomputed with the exact row maximum (all 48 scores of a
// query are in registers). Only the weights and the final state move through memory: one
// launch decodes every round and layer, and the readout follows on the state it writes.
//
// Four wavefronts (four windows) share one weight stream. The host lays each layer's weights
// out in the order the kernel consumes them, and the workgroup pulls the stream through a
// double-buffered LDS ring in chunks of 32 one-kilobyte fragments with direct global->LDS
// loads, spread between the current chunk's fragment reads. Per layer: for each 32-feature
// group og of Q/K/V (one chunk at d_model 128), the Q, K and V fragments of the group, the
// attention of the group's heads, and the out-projection's k-step og, whose input is exactly
// that group's attention output (the projections read a bf16 copy of the layer input, so the
// out-projection accumulates into the state in place); then LayerNorm 1, the feed-forward in
// chunks of 64 hidden units, and LayerNorm 2. A round is L (KS + F/64) chunks and the stream
// wraps from the last layer to the first, so the prefetch runs on across layers and rounds.
// Every fragment read from LDS feeds one MFMA per token block of the wavefront (TB of them).
#include "common.h"
#include "kernels.h"
#include "pipeline.h"

#include <type_traits>

namespace {

constexpr int FRAG = 512;          // bf16 values per fragment (1 KB)
constexpr int RWAVES = 4;          // wavefronts, i.e. windows, per workgroup
constexpr int RCHUNK = 32;         // fragments per ring buffer
constexpr int RD = 128;            // d_model of the resident path
constexpr int RRT = RD / 16;       // 16-row C tiles of a d_model vector
constexpr int RKS = RD / 32;       // 32-deep k-steps of a d_model vector
constexpr int RLA = 8;             // fragment reads in flight ahead of their MFMAs (8: 8% faster than 4 at d7)
constexpr int RMAXL = 4;           // layers whose vectors fit the LDS table

template <int MR>
struct RShape {
    static constexpr int F = MR * RD;
    static constexpr int CH = 64;                          // hidden units per feed-forward chunk
    static constexpr int NMLP = F / CH;
    static constexpr int QKV_FRAGS = 3 * 2 * RKS;          // Q, K, V of one 32-feature group
    static constexpr int W1_FRAGS = (CH / 16) * RKS, W2_FRAGS = RRT * (CH / 32);
    static constexpr int LAYER_CHUNKS = RKS + NMLP;
    static_assert(QKV_FRAGS + RRT == RCHUNK, "a Q/K/V group and its out-projection k-step fill one chunk");
    static_assert(W1_FRAGS + W2_FRAGS == RCHUNK, "a feed-forward chunk fills one ring buffer");
    static_assert(RKS % 2 == 0 && LAYER_CHUNKS % 2 == 0, "ring parity repeats every layer");
};

// Per-layer vectors, in the order the host writes them: [b_q b_k b_v | b_o g1 be1 b2 g2 be2 | b1].
template <int MR>
struct RVec {
    static constexpr int BQ = 0, BK = RD, BV = 2 * RD, BO = 3 * RD, G1 = 4 * RD, BE1 = 5 * RD, B2 = 6 * RD,
                         G2 = 7 * RD, BE2 = 8 * RD, B1 = 9 * RD;
    static constexpr int PER_LAYER = 9 * RD + MR * RD;
};

// The two ring buffers, separate objects so the compiler can tell they never alias.
template <int PAR>
PWD_DEV uint16_t* rbuf() {
    __shared__ __align__(16) uint16_t buf[RCHUNK * FRAG];
    return buf;
}

// The weight stream of a round: chunk i of L * LAYER_CHUNKS at stream + i * RCHUNK fragments.
// While chunk i is in use, each wavefront loads its RCHUNK / RWAVES fragments of chunk i + 1
// (wrapping to the first chunk after the last) into the other buffer, one load after each of
// read RLA, RLA + 2, ... of the chunk's fragment reads.
struct Ring {
    const uint16_t* stream;
    int nchunks, wave, lane;
    static constexpr int PER_WAVE = RCHUNK / RWAVES;

    __device__ const uint16_t* next(int i) const {
        return stream + (size_t)(i + 1 < nchunks ? i + 1 : 0) * RCHUNK * FRAG;
    }
    template <int PAR>
    __device__ void part(const uint16_t* src, int j) const {
        const int f = wave * PER_WAVE + j;
        lds_load_1k(uniform_ptr(src + f * FRAG), lds_addr(rbuf<PAR>() + f * FRAG), lane);
    }
    // after fragment read r of the chunk whose successor is `src`, going to buffer PAR
    template <int PAR>
    __device__ void after_read(const uint16_t* src, int r) const {
        if (r >= RLA && (r - RLA) % 2 == 0 && (r - RLA) / 2 < PER_WAVE) part<PAR>(src, (r - RLA) / 2);
    }
    // Chunk in buffer PAR becomes visible to every wavefront: this wavefront's loads of it have
    // landed (no other vector memory operation is outstanding at a chunk boundary that must
    // not be waited for), then the barrier also frees the other buffer for the next chunk.
    template <int PAR>
    __device__ const uint16_t* sync() const {
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        return rbuf<PAR>();
    }
};
static_assert(RLA + 2 * (Ring::PER_WAVE - 1) < 3 * 2 * RKS, "the next chunk's loads go out during the Q/K/V reads");

PWD_DEV bf16x4 to_b4(f32x4 v) {
    bf16x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = (__bf16)v[i];
    return r;
}

// Softmax over the window's keys for NP independent (query block, head) pairs at once, so that
// their latencies overlap: scores s[p][kb] (keys 4g+i of key block kb as rows, this lane's
// query as the column), padding keys (index >= ntok, only ever in the last block) excluded.
// SHIFT: with the exact row maximum subtracted; otherwise exponentiated as they are. The
// probabilities, rounded to bf16, go to pb (the P^T operand); sum gets their column sum, taken
// on the matrix core from the same bf16 values (an A operand whose row 0 is all ones turns P^T
// into its column sums, in row 0 of the result), in every lane of the column, and inv 1 / sum.
template <bool SHIFT, int NP, int TB>
PWD_DEV void softmax_cols(f32x4 (&s)[NP][TB], bf16x4 (&pb)[NP][TB], float (&sum)[NP], float (&inv)[NP], int ntok,
                          int g, bf16x4 ones) {
    if (ntok < TB * 16) {   // wavefront-uniform: the last block holds padding keys
#pragma unroll
        for (int p = 0; p < NP; ++p)
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if ((TB - 1) * 16 + 4 * g + i >= ntok) s[p][TB - 1][i] = -INFINITY;
    }
    float mx[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) mx[p] = 0.f;
    if constexpr (SHIFT) {
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            mx[p] = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < TB; ++kb)
                mx[p] = fmaxf(mx[p], fmaxf(fmaxf(s[p][kb][0], s[p][kb][1]), fmaxf(s[p][kb][2], s[p][kb][3])));
        }
#pragma unroll
        for (int p = 0; p < NP; ++p) mx[p] = group_max(mx[p]);
    }
    f32x4 ls[NP];
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        ls[p] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < TB; ++kb) {
            f32x4 e;
#pragma unroll
            for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(SHIFT ? s[p][kb][i] - mx[p] : s[p][kb][i]);
            pb[p][kb] = to_b4(e);
            ls[p] = mfma16x16x16(ones, pb[p][kb], ls[p]);
        }
    }
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        sum[p] = row0_broadcast(ls[p][0]);
        inv[p] = __builtin_amdgcn_rcpf(sum[p]);
    }
}

// True (wavefront-uniform) when every column sum lies in [1e-30, 2^126] and every output value
// is finite (x * 0 is 0 for finite x and NaN otherwise): the unshifted softmax is then the exact
// one up to rounding. Otherwise the caller recomputes with the row maximum subtracted.
template <int NP>
PWD_DEV bool in_range(const float (&sum)[NP], const f32x4 (&o)[NP]) {
    bool ok = true;
#pragma unroll
    for (int p = 0; p < NP; ++p) {
        float chk = sum[p];
#pragma unroll
        for (int i = 0; i < 4; ++i) chk = fmaf(o[p][i], 0.f, chk);
        ok = ok && chk >= 1e-30f && chk <= 0x1p126f;
    }
    return __builtin_amdgcn_ballot_w64(!ok) == 0;
}

// LayerNorm over the d_model features of each token (biased variance, two passes) of the state
// plus `bias_in` (per feature, or null), in one pass over the state: the result, plus
// `bias_out` (or null), goes back to the state, and the result itself (without bias_out) as bf16
// B fragments to xb when `pack` is set -- the next matrix product's operand.
template <int TB>
PWD_DEV void ln_pack(f32x4 (&x)[RRT][TB], const float* bias_in, const float* gamma, const float* beta,
                     const float* bias_out, bf16x8 (&xb)[RKS][TB], bool pack, float eps, int g) {
    constexpr float inv_d = 1.0f / RD;
#pragma unroll
    for (int b = 0; b < TB; ++b) {
        f32x4 y[RRT];
        float s = 0.f;
#pragma unroll
        for (int rt = 0; rt < RRT; ++rt) {
            y[rt] = x[rt][b];
            if (bias_in) y[rt] += ld4(bias_in + rt * 16 + 4 * g);
            s += (y[rt][0] + y[rt][1]) + (y[rt][2] + y[rt][3]);
        }
        const float mean = group_sum(s) * inv_d;
        float v = 0.f;
#pragma unroll
        for (int rt = 0; rt < RRT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                y[rt][i] -= mean;
                v = fmaf(y[rt][i], y[rt][i], v);
            }
        const float rstd = rsqrtf(group_sum(v) * inv_d + eps);
#pragma unroll
        for (int rt = 0; rt < RRT; ++rt) {
            const f32x4 gm = ld4(gamma + rt * 16 + 4 * g);
            const f32x4 bt = ld4(beta + rt * 16 + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i) y[rt][i] = fmaf(y[rt][i] * rstd, gm[i], bt[i]);
        }
        if (pack)
#pragma unroll
            for (int ks = 0; ks < RKS; ++ks) xb[ks][b] = pack_b(y[2 * ks], y[2 * ks + 1]);
#pragma unroll
        for (int rt = 0; rt < RRT; ++rt) x[rt][b] = bias_out ? y[rt] + ld4(bias_out + rt * 16 + 4 * g) : y[rt];
    }
}

template <int TB, int MR, int DH>
__global__ __launch_bounds__(RWAVES * 64, 1) void resident_kernel(ResidentParams p) {
    using S = RShape<MR>;
    using V = RVec<MR>;
    static_assert(DH == 16 || DH == 32, "heads of 16 or 32");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    // a wavefront past the batch decodes the last window again (the weight ring needs every
    // wavefront at every barrier) and stores nothing
    const int win_raw = (int)blockIdx.x * RWAVES + wave;
    const bool live = win_raw < p.in.nwin;
    const int win = live ? win_raw : p.in.nwin - 1;

    Ring ring;
    ring.stream = p.stream;
    ring.nchunks = p.L * S::LAYER_CHUNKS;
    ring.wave = __builtin_amdgcn_readfirstlane(wave);
    ring.lane = lane;
    ring.template part<0>(p.stream, 0);   // chunk 0 into buffer 0 ...
#pragma unroll
    for (int j = 1; j < Ring::PER_WAVE; ++j) ring.template part<0>(p.stream, j);

    // ... while the per-layer vectors, b_e + PE of the window's blocks and w_e go to LDS
    __shared__ __align__(16) float vec[RMAXL * V::PER_LAYER];
    __shared__ __align__(16) float s0[TB * RRT * 256];
    __shared__ __align__(16) float we[RD];
    for (int i = threadIdx.x; i < p.L * V::PER_LAYER; i += RWAVES * 64) vec[i] = p.vecs[i];
    for (int i = threadIdx.x; i < TB * RRT * 256; i += RWAVES * 64) s0[i] = p.S0[i];
    for (int i = threadIdx.x; i < RD; i += RWAVES * 64) we[i] = p.we[i];
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // chunk 0 and the tables are in LDS ...
    __syncthreads();                                    // ... and visible to every wavefront

    const uint32_t* meas = p.in.meas + (int64_t)win * (p.in.W + 1) * p.in.words;
    const int type = p.in.types[win];
    int stab[TB];   // this lane's token's stabilizer in each block, or -1 (reads word 0)
    uint32_t m_prev[TB], m_cur[TB];   // its measurement words of rows t and t + 1
#pragma unroll
    for (int b = 0; b < TB; ++b) {
        const int s = b * 16 + col;
        stab[b] = s < p.ntok ? (p.tok_stab ? p.tok_stab[s] : s) : -1;
        const int wd = stab[b] >= 0 ? stab[b] >> 5 : 0;
        m_prev[b] = meas[wd];
        m_cur[b] = meas[p.in.words + wd];
    }

    bf16x4 ones;   // A operand with row 0 all ones: column sums on the matrix core
#pragma unroll
    for (int i = 0; i < 4; ++i) ones[i] = (__bf16)(col == 0 ? 1.0f : 0.0f);

    f32x4 x[RRT][TB];
    bf16x8 xb[RKS][TB];   // the current matrix product's operand: a bf16 copy of the state
#pragma unroll
    for (int rt = 0; rt < RRT; ++rt)
#pragma unroll
        for (int b = 0; b < TB; ++b) x[rt][b] = f32x4{0.f, 0.f, 0.f, 0.f};   // D_0 = 0

    for (int t = 0; t < p.in.W; ++t) {
        // ---- embedding of round t folded into the state: X = kappa (E_t w_e + b_e + PE + X)
        float ev[TB];
#pragma unroll
        for (int b = 0; b < TB; ++b) {
            const uint32_t w = event_from(m_prev[b], m_cur[b], t, type, p.in.b_left, p.in.d);
            ev[b] = stab[b] >= 0 ? (float)((w >> (stab[b] & 31)) & 1u) : 0.f;
            m_prev[b] = m_cur[b];
        }
#pragma unroll
        for (int b = 0; b < TB; ++b) {
            const bool real = b * 16 + col < p.ntok;
#pragma unroll
            for (int rt = 0; rt < RRT; ++rt) {
                const f32x4 sv = ld4(s0 + ((b * RRT + rt) * 64 + lane) * 4);
                const f32x4 wv = ld4(we + rt * 16 + 4 * g);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    x[rt][b][i] = p.kappa * ((real ? ev[b] * wv[i] + sv[i] : 0.f) + x[rt][b][i]);
            }
        }

        // the layer input as B fragments, the projections' operand (layers after the first get
        // it from the previous layer's LayerNorm 2)
#pragma unroll
        for (int ks = 0; ks < RKS; ++ks)
#pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        for (int l = 0; l < p.L; ++l) {
            const float* vl = vec + l * V::PER_LAYER;
            const int cbase = l * S::LAYER_CHUNKS;

            // ---- per 32-feature group: Q, K, V, attention of its heads, out-projection k-step.
            // Groups run in pairs (ring buffers 0 and 1) in a loop rather than fully unrolled,
            // which keeps the code, and its compile time, small.
            auto og_group = [&](auto parc, int og) {
                constexpr int PAR = decltype(parc)::value;
                const uint16_t* buf = ring.template sync<PAR>();
                if (PAR == 0 && og == 0 && l == 0 && t + 2 <= p.in.W) {
                    // the next round's measurement words, issued ahead of this chunk's weight
                    // loads so they have landed by the next chunk's wait
#pragma unroll
                    for (int b = 0; b < TB; ++b)
                        m_cur[b] = meas[(t + 2) * p.in.words + (stab[b] >= 0 ? stab[b] >> 5 : 0)];
                }
                const uint16_t* nx = ring.next(cbase + og);
                f32x4 q[2][TB], k[2][TB], v[2][TB];
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int f0 = og * 32 + hh * 16;
                    const f32x4 bq = ld4(vl + V::BQ + f0 + 4 * g), bk = ld4(vl + V::BK + f0 + 4 * g);
                    const float bvv = vl[V::BV + f0 + col];   // V tiles: features along columns
#pragma unroll
                    for (int b = 0; b < TB; ++b) {
                        q[hh][b] = bq;
                        k[hh][b] = bk;
                        v[hh][b] = f32x4{bvv, bvv, bvv, bvv};
                    }
                }
                // fragment r: part r / (2 KS) (Q, K, V), k-step (r / 2) % KS, row tile r % 2
                pipelined<S::QKV_FRAGS, RLA>(
                    [&](int r) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(buf + r * FRAG + lane * 8)); },
                    [&](int r, const bf16x8& a) {
                        const int part = r / (2 * RKS), ks = (r / 2) % RKS, hh = r % 2;
#pragma unroll
                        for (int b = 0; b < TB; ++b) {
                            if (part == 0) q[hh][b] = mfma16x16x32(a, xb[ks][b], q[hh][b]);
                            else if (part == 1) k[hh][b] = mfma16x16x32(a, xb[ks][b], k[hh][b]);
                            else v[hh][b] = mfma16x16x32(xb[ks][b], a, v[hh][b]);
                        }
                    },
                    [&](int r) { ring.template after_read<1 - PAR>(nx, r); });
                sched_pipeline<S::QKV_FRAGS, TB, RLA>();

                // attention of the group's heads: y[qb] = O^T of query block qb as a B fragment
                bf16x8 y[TB];
                bf16x4 vt[2][TB];   // V^T A operands per 16-feature tile and key block
#pragma unroll
                for (int hh = 0; hh < 2; ++hh)
#pragma unroll
                    for (int b = 0; b < TB; ++b) vt[hh][b] = to_b4(v[hh][b]);
                const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
                if constexpr (DH == 16) {   // two heads per group: features 16 hh .. 16 hh + 15
                    constexpr int NP = 2 * TB;   // pair p = query block p / 2, head p % 2
                    bf16x4 q4[2][TB], k4[2][TB];
#pragma unroll
                    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
                        for (int b = 0; b < TB; ++b) {
                            q4[hh][b] = to_b4(q[hh][b] * p.qscale);
                            k4[hh][b] = to_b4(k[hh][b]);
                        }
                    f32x4 o[NP];
                    float inv[NP];
                    auto attend = [&](auto shift) {
                        f32x4 s[NP][TB];
                        bf16x4 pb[NP][TB];
                        float sum[NP];
#pragma unroll
                        for (int pp = 0; pp < NP; ++pp)
#pragma unroll
                            for (int kb = 0; kb < TB; ++kb) s[pp][kb] = mfma16x16x16(k4[pp % 2][kb], q4[pp % 2][pp / 2], zero);
                        softmax_cols<decltype(shift)::value, NP, TB>(s, pb, sum, inv, p.ntok, g, ones);
#pragma unroll
                        for (int pp = 0; pp < NP; ++pp) {
                            o[pp] = zero;
#pragma unroll
                            for (int kb = 0; kb < TB; ++kb) o[pp] = mfma16x16x16(vt[pp % 2][kb], pb[pp][kb], o[pp]);
                        }
                        return in_range<NP>(sum, o);
                    };
                    if (!attend(std::false_type{})) attend(std::true_type{});
#pragma unroll
                    for (int qb = 0; qb < TB; ++qb) y[qb] = pack_b(o[2 * qb] * inv[2 * qb], o[2 * qb + 1] * inv[2 * qb + 1]);
                } else {   // one head of 32 features
                    bf16x8 qf[TB], kf[TB];
#pragma unroll
                    for (int b = 0; b < TB; ++b) {
                        qf[b] = pack_b(q[0][b] * p.qscale, q[1][b] * p.qscale);
                        kf[b] = pack_b(k[0][b], k[1][b]);
                    }
                    f32x4 o[TB][2];
                    float inv[TB];
                    auto attend = [&](auto shift) {
                        f32x4 s[TB][TB];
                        bf16x4 pb[TB][TB];
                        float sum[TB];
#pragma unroll
                        for (int qb = 0; qb < TB; ++qb)
#pragma unroll
                            for (int kb = 0; kb < TB; ++kb) s[qb][kb] = mfma16x16x32(kf[kb], qf[qb], zero);
                        softmax_cols<decltype(shift)::value, TB, TB>(s, pb, sum, inv, p.ntok, g, ones);
#pragma unroll
                        for (int qb = 0; qb < TB; ++qb)
#pragma unroll
                            for (int hh = 0; hh < 2; ++hh) {
                                o[qb][hh] = zero;
#pragma unroll
                                for (int kb = 0; kb < TB; ++kb) o[qb][hh] = mfma16x16x16(vt[hh][kb], pb[qb][kb], o[qb][hh]);
                            }
                        // both halves of each query block's output against its sum
                        float sum2[2 * TB];
                        f32x4 o2[2 * TB];
#pragma unroll
                        for (int qb = 0; qb < TB; ++qb)
#pragma unroll
                            for (int hh = 0; hh < 2; ++hh) {
                                sum2[2 * qb + hh] = sum[qb];
                                o2[2 * qb + hh] = o[qb][hh];
                            }
                        return in_range<2 * TB>(sum2, o2);
                    };
                    if (!attend(std::false_type{})) attend(std::true_type{});
#pragma unroll
                    for (int qb = 0; qb < TB; ++qb) y[qb] = pack_b(o[qb][0] * inv[qb], o[qb][1] * inv[qb]);
                }

                // out-projection k-step og: X += Wo[:, og]^T y (the residual is the state itself)
                pipelined<RRT, RLA>(
                    [&](int r) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(buf + (S::QKV_FRAGS + r) * FRAG + lane * 8)); },
                    [&](int r, const bf16x8& a) {
#pragma unroll
                        for (int b = 0; b < TB; ++b) x[r][b] = mfma16x16x32(a, y[b], x[r][b]);
                    },
                    [](int) {});
                sched_pipeline<RRT, TB, RLA>();
            };
            for (int og = 0; og < RKS; og += 2) {
                og_group(std::integral_constant<int, 0>{}, og);
                og_group(std::integral_constant<int, 1>{}, og + 1);
            }
            // LayerNorm 1 of X + b_o; its output is the feed-forward's operand, and the
            // feed-forward accumulators start at that output + b_2
            ln_pack<TB>(x, vl + V::BO, vl + V::G1, vl + V::BE1, vl + V::B2, xb, true, p.eps, g);

            // ---- feed-forward in chunks of 64 hidden units
            constexpr int NRH = S::CH / 16, NKH = S::CH / 32;
            auto mlp_chunk = [&](auto parc, int c) {
                constexpr int PAR = decltype(parc)::value;   // = (KS + c) & 1, KS even
                const uint16_t* buf = ring.template sync<PAR>();
                const uint16_t* nx = ring.next(cbase + RKS + c);
                f32x4 h[NRH][TB];
#pragma unroll
                for (int rh = 0; rh < NRH; ++rh) {
                    const f32x4 b1 = ld4(vl + V::B1 + c * S::CH + rh * 16 + 4 * g);
#pragma unroll
                    for (int b = 0; b < TB; ++b) h[rh][b] = b1;
                }
                bf16x8 hb[NKH][TB];
                // W1 fragment r: k-step r / NRH, hidden row tile r % NRH; then W2 fragment
                // r - W1_FRAGS: hidden k-step (r - W1) / RT, output row tile (r - W1) % RT
                pipelined<RCHUNK, RLA>(
                    [&](int r) { return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(buf + r * FRAG + lane * 8)); },
                    [&](int r, const bf16x8& a) {
                        if (r < S::W1_FRAGS) {
                            const int ks = r / NRH, rh = r % NRH;
#pragma unroll
                            for (int b = 0; b < TB; ++b) h[rh][b] = mfma16x16x32(a, xb[ks][b], h[rh][b]);
                            if (r == S::W1_FRAGS - 1) {
#pragma unroll
                                for (int kh = 0; kh < NKH; ++kh)
#pragma unroll
                                    for (int b = 0; b < TB; ++b) {
                                        f32x4 lo = h[2 * kh][b], hi = h[2 * kh + 1][b];
#pragma unroll
                                        for (int i = 0; i < 4; ++i) {
                                            lo[i] = fmaxf(lo[i], 0.f);
                                            hi[i] = fmaxf(hi[i], 0.f);
                                        }
                                        hb[kh][b] = pack_b(lo, hi);
                                    }
                            }
                        } else {
                            const int kh = (r - S::W1_FRAGS) / RRT, rt = (r - S::W1_FRAGS) % RRT;
#pragma unroll
                            for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, hb[kh][b], x[rt][b]);
                        }
                    },
                    [&](int r) { ring.template after_read<1 - PAR>(nx, r); });
                sched_pipeline<RCHUNK, TB, RLA>();
            };
            static_assert(S::NMLP % 2 == 0, "feed-forward chunks in pairs");
            for (int c = 0; c < S::NMLP; c += 2) {
                mlp_chunk(std::integral_constant<int, 0>{}, c);
                mlp_chunk(std::integral_constant<int, 1>{}, c + 1);
            }
            // LayerNorm 2; its output is the next layer's operand (the last layer's is the state
            // D_t, which the next round's embedding changes first)
            ln_pack<TB>(x, nullptr, vl + V::G2, vl + V::BE2, nullptr, xb, l + 1 < p.L, p.eps, g);
        }
    }

    // the final state D_W for the readout
    if (live) {
#pragma unroll
        for (int b = 0; b < TB; ++b)
#pragma unroll
            for (int rt = 0; rt < RRT; ++rt)
                *reinterpret_cast<f32x4*>(p.X + ((((int64_t)win * p.nbw + b) * RRT + rt) * 64 + lane) * 4) = x[rt][b];
    }
    // the last chunk's prefetch (the first chunk again) lands before the LDS is freed
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

template <int TB, int MR>
hipError_t launch_tb_mr(int dh, const ResidentParams& p, hipStream_t s) {
    const dim3 grid((unsigned)((p.in.nwin + RWAVES - 1) / RWAVES)), block(RWAVES * 64);
    if (dh == 16) resident_kernel<TB, MR, 16><<<grid, block, 0, s>>>(p);
    else if (dh == 32) resident_kernel<TB, MR, 32><<<grid, block, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

template <int TB>
hipError_t launch_tb(int mr, int dh, const ResidentParams& p, hipStream_t s) {
    if (mr == 4) return launch_tb_mr<TB, 4>(dh, p, s);
    return hipErrorInvalidValue;
}

}  // namespace

bool resident_supported(int D, int nbw, int L, int mr, int dh) {
    return D == RD && nbw >= 1 && nbw <= 4 && L >= 1 && L <= RMAXL && mr == 4 && (dh == 16 || dh == 32);
}

int resident_chunk_fragments() { return RCHUNK; }

hipError_t launch_resident(int mr, int dh, const ResidentParams& p, hipStream_t s) {
    if (p.in.nwin <= 0) return hipSuccess;
    switch (p.nbw) {
        case 1: return launch_tb<1>(mr, dh, p, s);
        case 2: return launch_tb<2>(mr, dh, p, s);
        case 3: return launch_tb<3>(mr, dh, p, s);
        case 4: return launch_tb<4>(mr, dh, p, s);
        default: return hipErrorInvalidValue;
    }
}
