// Building blocks shared by the kernels that stream weight fragments through LDS: the
// software-pipelined fragment reader, its scheduling request, a compile-time loop and the
// LayerNorm over the features of each token held as MFMA C fragments.
#pragma once
#include "common.h"

#include <type_traits>
#include <utility>

namespace {

PWD_DEV f32x4 ld4(const float* __restrict__ p) { return *reinterpret_cast<const f32x4*>(p); }

// The fragment reads of one chunk, software-pipelined in program order: LA reads are in
// flight ahead of the MFMAs; read r + LA is issued right after the MFMAs that consume read
// r. read(r) loads fragment r of the chunk, use(r, a) issues the MFMAs of fragment r, and
// after(r) runs right after read r is issued. Every loop is fully unrolled, so the ring
// indices are compile-time constants and the ring lives in registers.
template <int NREAD, int LA, typename Read, typename Use, typename After>
PWD_DEV void pipelined(const Read& read, const Use& use, const After& after) {
    static_assert(LA >= 1 && LA <= NREAD, "look-ahead");
    bf16x8 ring[LA];
#pragma unroll
    for (int r = 0; r < LA; ++r) {
        ring[r] = read(r);
        after(r);
    }
#pragma unroll
    for (int r = 0; r < NREAD; ++r) {
        use(r, ring[r % LA]);
        if (r + LA < NREAD) {
            ring[r % LA] = read(r + LA);
            after(r + LA);
        }
    }
}

// Keeps the scheduler on the program order above: LA reads, then (MPR MFMAs, one read)
// pairs, then the MFMAs of the last LA fragments.
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

template <typename F, int... I>
PWD_DEV void static_for_impl(const F& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
// f(integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time
template <int N, typename F>
PWD_DEV void static_for(const F& f) { static_for_impl(f, std::make_integer_sequence<int, N>{}); }

// As sched_pipeline, for chunks whose first NPAIRED reads come in pairs (the two halves of one
// 8-bit fragment): the MFMAs of a pair follow its second read.
template <int NREAD, int MPR, int LA, int NPAIRED>
PWD_DEV void sched_pipeline_pairs() {
    static_assert(NPAIRED % 2 == 0 && NPAIRED <= NREAD, "whole pairs");
    constexpr auto mfmas = [](int r) { return r < NPAIRED ? (r & 1 ? MPR : 0) : MPR; };
    __builtin_amdgcn_sched_group_barrier(0x100, LA, 0);
    static_for<NREAD - LA>([&](auto kc) {
        constexpr int M = mfmas(decltype(kc)::value);
        if constexpr (M > 0) __builtin_amdgcn_sched_group_barrier(0x008, M, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    });
    constexpr int TAIL = [=] {
        int n = 0;
        for (int k = NREAD - LA; k < NREAD; ++k) n += mfmas(k);
        return n;
    }();
    __builtin_amdgcn_sched_group_barrier(0x008, TAIL, 0);
}

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

}  // namespace
