// Stream decoding around decode_windows: cutting a memory experiment into overlapping
// windows (Sec. 3.1) and combining the per-window results into the global correction
// (eq. global_xor) and its soft probability (eq. soft_xor).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int SPLIT_THREADS = 256;
constexpr int COMBINE_THREADS = 256;

// One thread per (window, row, word): meas[i][k][w] = R[i d - b_left - 1 + k][w], zero
// before the stream and R[T-1] after it. Consecutive threads copy consecutive words. The
// index arithmetic is 32-bit (IDX = uint32_t) whenever the output has fewer than 2^31 words.
template <typename IDX>
__global__ __launch_bounds__(SPLIT_THREADS) void stream_split_kernel(StreamSplitParams p) {
    const IDX idx = (IDX)blockIdx.x * SPLIT_THREADS + threadIdx.x;
    const IDX total = (IDX)p.m * (IDX)(p.W + 1) * (IDX)p.words;
    if (idx < total) {
        const IDX r = idx / (IDX)p.words;
        const int w = (int)(idx - r * (IDX)p.words);
        const IDX i = r / (IDX)(p.W + 1);
        const int k = (int)(r - i * (IDX)(p.W + 1));
        const int64_t src = (int64_t)i * p.d - p.b_left - 1 + k;
        p.meas[idx] = src < 0 ? 0u : p.stream[(src < p.T ? src : p.T - 1) * p.words + w];
    }
    if (idx < (IDX)p.m) p.types[idx] = idx == 0 ? WIN_INITIAL : (idx == (IDX)p.m - 1 ? WIN_FINAL : WIN_BULK);
}

// One workgroup: XOR of the window bits and prod_k (1 - 2 sigmoid(logit_k)) in double (and,
// when asked for, each window's probability sigmoid(logit_k) rounded to float). Each
// thread takes a fixed stride of windows and the partial results are combined by a fixed
// tree, so the result does not depend on timing.
__global__ __launch_bounds__(COMBINE_THREADS) void stream_combine_kernel(StreamCombineParams p) {
    __shared__ double prod[COMBINE_THREADS];
    __shared__ int parity[COMBINE_THREADS];
    double pr = 1.0;
    int x = 0;
    for (int i = threadIdx.x; i < p.m; i += COMBINE_THREADS) {
        const double y = 1.0 / (1.0 + exp(-(double)p.logits[i]));
        if (p.probs) p.probs[i] = (float)y;
        pr *= 1.0 - 2.0 * y;
        x ^= p.bits[i] & 1;
    }
    prod[threadIdx.x] = pr;
    parity[threadIdx.x] = x;
    __syncthreads();
    for (int n = COMBINE_THREADS / 2; n > 0; n >>= 1) {
        if ((int)threadIdx.x < n) {
            prod[threadIdx.x] *= prod[threadIdx.x + n];
            parity[threadIdx.x] ^= parity[threadIdx.x + n];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *p.bit = (uint8_t)parity[0];
        if (p.prob) *p.prob = (float)(0.5 * (1.0 - prod[0]));
    }
}

}  // namespace

hipError_t launch_stream_split(const StreamSplitParams& p, hipStream_t s) {
    const int64_t total = (int64_t)p.m * (p.W + 1) * p.words;
    const int64_t n = total > p.m ? total : p.m;
    const dim3 grid((unsigned)((n + SPLIT_THREADS - 1) / SPLIT_THREADS)), block(SPLIT_THREADS);
    if (n < ((int64_t)1 << 31)) stream_split_kernel<uint32_t><<<grid, block, 0, s>>>(p);
    else stream_split_kernel<uint64_t><<<grid, block, 0, s>>>(p);
    return hipGetLastError();
}

hipError_t launch_stream_combine(const StreamCombineParams& p, hipStream_t s) {
    stream_combine_kernel<<<dim3(1), dim3(COMBINE_THREADS), 0, s>>>(p);
    return hipGetLastError();
}
