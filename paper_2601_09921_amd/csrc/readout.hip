// Readout of the final decoder state (App. A.3) and the detection-event export.
//
// Readout, one workgroup per window, one thread per output feature o:
//   the tokens go back onto the (d+1)x(d+1) stabilizer grid (zeros at empty cells);
//   Y[i][j] = ReLU(b_c + sum_{a,b in {0,1}} G[i+a][j+b] Wc[a][b])  (2x2 valid convolution)
//   P[i] = mean_j Y[i][j]                                           (logical pooling)
//   logit = sum_i <w_o[i], P[i]> + b_o + beta[type],  bit = logit > 0
// in fp32, two data-qubit rows at a time with three grid rows staged in LDS. The final sum
// over features is a fixed-order tree, so a window's logit does not depend on the batch.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int MAXD = 25;
constexpr int ROWS = 2;      // data-qubit rows per pass

__global__ __launch_bounds__(256) void readout_kernel(ReadoutParams p) {
    const int win = blockIdx.x;
    const int o = threadIdx.x;            // output feature (blockDim.x == D)
    const int D = p.D, d = p.d, gw = d + 1;
    extern __shared__ __align__(16) float gsh[];   // [ROWS+1][d+1][D]
    __shared__ float red[256];

    const int type = p.types[win];
    const bool bad = type > WIN_FINAL;
    const int RT = D / 16;
    const int64_t tb_base = (int64_t)win * p.nbw;

    float part = 0.f;
    for (int i0 = 0; i0 < d; i0 += ROWS) {
        const int nrow = min(ROWS, d - i0);
        __syncthreads();
        // stage grid rows i0 .. i0+nrow into LDS (thread o moves feature o of each cell)
        for (int r = 0; r <= nrow; ++r)
            for (int c = 0; c < gw; ++c) {
                const int tok = p.cell_token[(i0 + r) * gw + c];
                float v = 0.f;
                if (tok >= 0) {
                    const int blk = tok >> 4, cl = tok & 15;
                    const int rt = o >> 4, g = (o & 15) >> 2, i = o & 3;
                    v = p.X[(((tb_base + blk) * RT + rt) * 64 + g * 16 + cl) * 4 + i];
                }
                gsh[(r * gw + c) * D + o] = v;
            }
        __syncthreads();
        float acc[ROWS][MAXD];
        const float bias = p.bc[o];
#pragma unroll
        for (int r = 0; r < ROWS; ++r)
#pragma unroll
            for (int j = 0; j < MAXD; ++j) acc[r][j] = bias;
        for (int a = 0; a < 2; ++a)
            for (int b = 0; b < 2; ++b)
                for (int k = 0; k < D; ++k) {
                    const float wv = p.Wc[(((a * 2 + b) * D) + k) * D + o];
#pragma unroll
                    for (int r = 0; r < ROWS; ++r) {
                        const float* grow = gsh + ((r + a) * gw + b) * D + k;
#pragma unroll
                        for (int j = 0; j < MAXD; ++j)
                            if (r < nrow && j < d) acc[r][j] = fmaf(grow[j * D], wv, acc[r][j]);
                    }
                }
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
            if (r >= nrow) continue;
            float pool = 0.f;
#pragma unroll
            for (int j = 0; j < MAXD; ++j)
                if (j < d) pool += fmaxf(acc[r][j], 0.f);
            part = fmaf(p.wo[(i0 + r) * D + o], pool / (float)d, part);
        }
    }
    red[o] = part;
    __syncthreads();
    for (int n = 128; n > 0; n >>= 1) {
        if (o < n && o + n < D) red[o] += red[o + n];
        __syncthreads();
    }
    if (o == 0) {
        if (bad) {
            p.logits[win] = __builtin_nanf("");
            p.bits[win] = 0;
            atomicOr(p.err, 1);
        } else {
            const float logit = red[0] + p.bo + p.beta[type];
            p.logits[win] = logit;
            p.bits[win] = logit > 0.f ? 1 : 0;
        }
    }
}

__global__ void events_kernel(EventsParams p) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t per_win = (int64_t)p.in.W * p.in.words;
    if (idx >= per_win * p.in.nwin) return;
    const int64_t win = idx / per_win;
    const int rem = (int)(idx - win * per_win);
    const int t = rem / p.in.words, wd = rem % p.in.words;
    const int type = p.in.types[win];
    uint32_t e = 0u;
    if (type > WIN_FINAL) {
        atomicOr(p.err, 1);
    } else {
        e = event_word(p.in.meas + win * (int64_t)(p.in.W + 1) * p.in.words, p.in.words, t, wd,
                       type, p.in.b_left, p.in.d);
        const int valid = p.in.N - wd * 32;
        if (valid < 32) e &= (1u << valid) - 1u;
    }
    p.events[idx] = e;
}

}  // namespace

hipError_t launch_readout(const ReadoutParams& p, hipStream_t s) {
    if (p.nwin <= 0) return hipSuccess;
    if (p.d > MAXD || p.D > 256) return hipErrorInvalidValue;
    const size_t smem = (size_t)(ROWS + 1) * (p.d + 1) * p.D * sizeof(float);
    hipError_t e = hipFuncSetAttribute((const void*)readout_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    readout_kernel<<<dim3((unsigned)p.nwin), dim3(p.D), smem, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_events(const EventsParams& p, hipStream_t s) {
    const int64_t total = (int64_t)p.in.nwin * p.in.W * p.in.words;
    if (total <= 0) return hipSuccess;
    events_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s>>>(p);
    return hipGetLastError();
}
