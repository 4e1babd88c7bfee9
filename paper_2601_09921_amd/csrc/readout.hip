// Readout of the final decoder state (App. A.3) and the detection-event export.
//
// Readout:
//   the tokens go back onto the (d+1)x(d+1) stabilizer grid (zeros at empty cells);
//   Y[i][j] = ReLU(b_c + sum_{a,b in {0,1}} G[i+a][j+b] Wc[a][b])  (2x2 valid convolution)
//   P[i] = mean_j Y[i][j]                                           (logical pooling)
//   logit = sum_i <w_o[i], P[i]> + b_o + beta[type],  bit = logit > 0
// The convolution is an implicit GEMM on bf16 MFMA (state rounded to bf16, fp32
// accumulation); pooling and the projection fold into one fixed-order sum, so a window's
// logit does not depend on the batch.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int RWAVES = 4;
constexpr int PB = 8;          // 16-position blocks per workgroup pass (128 positions)

PWD_DEV f32x4 ld4g(const float* __restrict__ p) { return *reinterpret_cast<const f32x4*>(p); }

// One workgroup per window. The d x d output positions (data qubits) form 16-wide MFMA
// column blocks; Y^T = Wc^T G^T over k = 4 taps x D input features, where the B fragment of
// (tap (a,b), features 32s..32s+31) holds the state of the stabilizer at cell (i+a, j+b)
// rounded to bf16 (zero where the cell is empty). A pass covers PB position blocks: for each
// tap the workgroup gathers their B fragments into LDS once, and each wavefront multiplies
// them by the A fragments (from L2) of its quarter of the output features, so every weight
// fragment feeds PB MFMAs and every gathered fragment feeds D / 64 of each wavefront. Each
// lane then adds sum_o w_o[i][o] ReLU(Y[o] + b_c[o]) / d over its outputs; one fixed-order
// reduction over lanes and wavefronts gives the window's sum.
template <int D>
__global__ __launch_bounds__(RWAVES * 64, 2) void readout_kernel(ReadoutParams p) {
    constexpr int RT = D / 16, KSD = D / 32, KS = 4 * KSD;
    constexpr int RTW = RT / RWAVES;                  // output row tiles per wavefront
    constexpr int GPB = PB / RWAVES;                  // position blocks gathered per wavefront
    static_assert(RT % RWAVES == 0 && PB % RWAVES == 0, "whole tiles per wavefront");
    const int win = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int d = p.d, gw = d + 1, npos = d * d, npb = (npos + 15) / 16;
    const int64_t tb_base = (int64_t)win * p.nbw;
    const float inv_d = 1.0f / (float)d;
    __shared__ __align__(16) uint16_t bsm[PB * KSD * 512];   // [PB][KSD] gathered B fragments
    __shared__ float red[RWAVES];

    // gathered B fragment of token T (-1: empty cell), features 32 s .. 32 s + 31
    auto gather = [&](int T, int s) -> u16x8 {
        u16x8 v = {0, 0, 0, 0, 0, 0, 0, 0};
        if (T < 0) return v;
        if (p.Xb) {   // bf16 state: the rounded values the fp32 branch computes
            const uint16_t* src = p.Xb + ((tb_base + (T >> 4)) * RT + 2 * s) * 256 + (g * 16 + (T & 15)) * 4;
            const u16x4 l4 = *reinterpret_cast<const u16x4*>(src);
            const u16x4 h4 = *reinterpret_cast<const u16x4*>(src + 256);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = l4[i];
                v[4 + i] = h4[i];
            }
            return v;
        }
        const float* src = p.X + ((tb_base + (T >> 4)) * RT + 2 * s) * 256 + (g * 16 + (T & 15)) * 4;
        return __builtin_bit_cast(u16x8, pack_b(ld4g(src), ld4g(src + 256)));
    };

    float part = 0.f;
    for (int pb0 = 0; pb0 < npb; pb0 += PB) {
        f32x4 acc[RTW][PB];
#pragma unroll
        for (int rr = 0; rr < RTW; ++rr)
#pragma unroll
            for (int b = 0; b < PB; ++b) acc[rr][b] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int t = 0; t < 4; ++t) {
            // this wavefront's GPB position blocks of the pass, every k-step of tap t
#pragma unroll
            for (int q = 0; q < GPB; ++q) {
                const int pbl = wave * GPB + q;
                const int pos = (pb0 + pbl) * 16 + col;
                int T = -1;
                if (pos < npos) {
                    const int i = pos / d, j = pos % d;
                    T = p.cell_token[(i + (t >> 1)) * gw + j + (t & 1)];
                }
#pragma unroll
                for (int s = 0; s < KSD; ++s)
                    *reinterpret_cast<u16x8*>(bsm + ((pbl * KSD + s) * 64 + lane) * 8) = gather(T, s);
            }
            __syncthreads();
#pragma unroll 2
            for (int s = 0; s < KSD; ++s) {
                bf16x8 a[RTW];
#pragma unroll
                for (int rr = 0; rr < RTW; ++rr)
                    a[rr] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(
                        p.Wc + (((size_t)(wave * RTW + rr) * KS + t * KSD + s) * 64 + lane) * 8));
#pragma unroll
                for (int b = 0; b < PB; ++b) {
                    const bf16x8 bb = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(
                        bsm + ((b * KSD + s) * 64 + lane) * 8));
#pragma unroll
                    for (int rr = 0; rr < RTW; ++rr) acc[rr][b] = mfma16x16x32(a[rr], bb, acc[rr][b]);
                }
            }
            __syncthreads();   // the next tap's gather overwrites the fragments
        }
#pragma unroll
        for (int b = 0; b < PB; ++b) {
            const int pos = (pb0 + b) * 16 + col;
            if (pos >= npos) continue;
            const float* wrow = p.wo + (pos / d) * D;
            float sum = 0.f;
#pragma unroll
            for (int rr = 0; rr < RTW; ++rr) {
                const int o = (wave * RTW + rr) * 16 + 4 * g;
                const f32x4 bias = ld4g(p.bc + o);
                const f32x4 w = ld4g(wrow + o);
#pragma unroll
                for (int i = 0; i < 4; ++i) sum = fmaf(w[i], fmaxf(acc[rr][b][i] + bias[i], 0.f), sum);
            }
            part += sum * inv_d;
        }
    }
    // fixed-order reduction: lanes, then wavefronts
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) part += __shfl_xor(part, off);
    if (lane == 0) red[wave] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
        float tot = 0.f;
#pragma unroll
        for (int w = 0; w < RWAVES; ++w) tot += red[w];
        const int type = p.types[win];
        const int64_t o = (int64_t)win * p.stride;
        if (type > WIN_FINAL) {
            p.logits[o] = __builtin_nanf("");
            p.bits[o] = 0;
            atomicOr(p.err, 1);
        } else {
            const float logit = tot + p.bo + p.beta[type];
            p.logits[o] = logit;
            p.bits[o] = logit > 0.f ? 1 : 0;
        }
    }
}

// One thread per output word; 32-bit index arithmetic (IDX = uint32_t) below 2^31 words.
template <typename IDX>
__global__ void events_kernel(EventsParams p) {
    const IDX idx = (IDX)blockIdx.x * blockDim.x + threadIdx.x;
    const IDX per_win = (IDX)p.in.W * (IDX)p.in.words;
    if (idx >= per_win * (IDX)p.in.nwin) return;
    const IDX win = idx / per_win;
    const int rem = (int)(idx - win * per_win);
    const int t = rem / p.in.words, wd = rem - t * p.in.words;
    const int type = p.in.types[win];
    uint32_t e = 0u;
    if (type > WIN_FINAL) {
        atomicOr(p.err, 1);
    } else {
        e = event_word(p.in.meas + (int64_t)win * (p.in.W + 1) * p.in.words, p.in.words, t, wd,
                       type, p.in.b_left, p.in.d);
        const int valid = p.in.N - wd * 32;
        if (valid < 32) e &= (1u << valid) - 1u;
    }
    p.events[idx] = e;
}

}  // namespace

hipError_t launch_readout(const ReadoutParams& p, hipStream_t s) {
    if (p.nwin <= 0) return hipSuccess;
    const dim3 grid((unsigned)p.nwin), block(RWAVES * 64);
    if (p.D == 256) readout_kernel<256><<<grid, block, 0, s>>>(p);
    else if (p.D == 128) readout_kernel<128><<<grid, block, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_events(const EventsParams& p, hipStream_t s) {
    const int64_t total = (int64_t)p.in.nwin * p.in.W * p.in.words;
    if (total <= 0) return hipSuccess;
    const dim3 grid((unsigned)((total + 255) / 256)), block(256);
    if (total < ((int64_t)1 << 31)) events_kernel<uint32_t><<<grid, block, 0, s>>>(p);
    else events_kernel<uint64_t><<<grid, block, 0, s>>>(p);
    return hipGetLastError();
}
