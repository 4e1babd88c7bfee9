// Multi-head self-attention across the stabilizer tokens of each window (App. A.2; the
// model table's Multi-Head Attention), bf16 MFMA with fp32 softmax statistics.
//
// One workgroup per (window, head), of 1, 2 or 4 wavefronts by window size. K_h and V_h are
// copied to LDS once, by direct global->LDS loads of the fragments the Q/K/V projection wrote
// (K as B fragments of K^T, which serve as A fragments of K; V as 16x16 tiles with tokens as
// rows, whose per-lane halves of two key blocks form an A fragment of V^T); each wavefront
// then takes its quarter of the
// 16-query blocks, four (the last pass two) at a time, and streams the keys in steps of 32:
//   S^T = K Q'^T - m      (16 keys x 16 queries per MFMA, lanes hold queries)
//   P^T = exp2(S^T)       (P^T is the S^T accumulator rounded to bf16, no shuffle)
//   O^T += V^T P^T,  l += 1^T P^T
// Q' = Q log2(e)/sqrt(dh) comes pre-scaled from the Q/K/V projection, so S is in log2 units.
// The shift m of a query is the Cauchy-Schwarz bound |q'| max_k |k| >= every score of the
// row; softmax is shift-invariant, so this is the exact softmax without a running maximum
// or rescaling, and m enters as the initial value of the MFMA accumulator. Should a row's
// sum underflow (a bound far above the true maximum), that query block is recomputed with
// the running-maximum form. Padding keys (index >= N) get probability 0. The row sums l come
// from the matrix core too: an A fragment whose row 0 is all ones turns P^T into its column
// sums, so numerator and denominator use the same bf16 probabilities and the VALU is left to
// the exponentials. The output is written as the B fragments the out-projection consumes.
#include "common.h"
#include "kernels.h"

namespace {

#ifndef ATTN_QMAX
#define ATTN_QMAX 4
#endif
constexpr int QMAX = ATTN_QMAX;       // query blocks per wavefront pass (the last takes QMAX / 2)
constexpr int SBATCH = 10;            // key blocks per wavefront per staging batch (d=25: one batch)

PWD_DEV float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

template <int DH>
struct Frag;
template <>
struct Frag<32> {
    using T = bf16x8;
    static __device__ __forceinline__ f32x4 mma(T a, T b, f32x4 c) { return mfma16x16x32(a, b, c); }
};
template <>
struct Frag<16> {
    using T = bf16x4;
    static __device__ __forceinline__ f32x4 mma(T a, T b, f32x4 c) { return mfma16x16x16(a, b, c); }
};

// K fragment of key block kb (LDS holds whole 1 KB fragments; with dh = 16 one fragment
// carries two heads and slot0 selects this head's four values).
template <int DH>
PWD_DEV typename Frag<DH>::T ld_kfrag(const uint16_t* ks, int kb, int lane, int slot0) {
    if constexpr (DH == 32)
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(ks + (kb * 64 + lane) * 8));
    else
        return __builtin_bit_cast(bf16x4, *reinterpret_cast<const u16x4*>(ks + (kb * 64 + lane) * 8 + slot0));
}

// V^T A fragment of the 32 keys of superblock sb for dh columns 16 half .. 16 half + 15: this
// lane's four keys of key block 2 sb (k slots 0-3) and of key block 2 sb + 1 (k slots 4-7),
// i.e. the lane's 8 bytes of tile half `half` of both V fragments.
PWD_DEV bf16x8 ld_vfrag(const uint16_t* vs, int half, int sb, int lane) {
    const uint16_t* t = vs + (2 * sb) * 512 + half * 256 + lane * 4;
    const u16x4 lo = *reinterpret_cast<const u16x4*>(t);
    const u16x4 hi = *reinterpret_cast<const u16x4*>(t + 512);
    u16x8 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[i] = lo[i];
        v[4 + i] = hi[i];
    }
    return __builtin_bit_cast(bf16x8, v);
}

PWD_DEV float sum4(float v) {
    v += __shfl_xor(v, 16);
    return v + __shfl_xor(v, 32);
}

template <int DH, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void attn_kernel(AttnParams p) {
    using FT = typename Frag<DH>::T;
    constexpr int RT = DH / 16;                 // 16-row tiles of O^T
    constexpr int NV = DH == 32 ? 8 : 4;        // Q/K values per lane
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int win = blockIdx.x / p.H, h = blockIdx.x % p.H;
    const int nbw = p.nbw, N = p.N;
    const int KSD = p.H * DH / 32;              // fragments per Q/K/V of a token block
    const int64_t tb_base = (int64_t)win * nbw;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem);   // [nbw][512]: K fragments
    uint16_t* vs = ks + (size_t)nbw * 512;               // [nbw + 1][512]: V tiles, + a zero block
    __shared__ float kmax_w[WAVES];

    // fragment and slot range of head h inside a Q/K/V fragment
    const int frag = DH == 32 ? h : h / 2;
    const int slot0 = DH == 32 ? 0 : (h % 2) * 4;
    const int vhalf = DH == 32 ? 0 : h % 2;     // V tile half of this head (dh = 16)

    // ---- stage K and V: one 1 KB direct load per fragment; an odd key-block count gets a
    // zero V block so the last superblock's missing keys meet P = 0 and V = 0
    for (int kb = wave; kb < nbw; kb += WAVES) {
        const uint16_t* src = p.QKV + (((tb_base + kb) * 3 + 1) * KSD + frag) * 512;
        lds_load_1k(uniform_ptr(src), lds_addr(ks + kb * 512), lane);
        lds_load_1k(uniform_ptr(src + KSD * 512), lds_addr(vs + kb * 512), lane);
    }
    if (nbw & 1)
        for (int i = threadIdx.x; i < 256; i += blockDim.x) reinterpret_cast<uint32_t*>(vs + nbw * 512)[i] = 0u;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // max |k| over the real keys
    float kmax2 = 0.f;
    for (int kb = wave; kb < nbw; kb += WAVES) {
        const u16x8 kv = *reinterpret_cast<const u16x8*>(ks + (kb * 64 + lane) * 8);
        float n2 = 0.f;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const float f = (float)__builtin_bit_cast(__bf16, (uint16_t)kv[slot0 + i]);
            n2 = fmaf(f, f, n2);
        }
        n2 = sum4(n2);
        if (kb * 16 + col < N) kmax2 = fmaxf(kmax2, n2);
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) kmax2 = fmaxf(kmax2, __shfl_xor(kmax2, off));
    if (lane == 0) kmax_w[wave] = kmax2;
    __syncthreads();
    float kmax = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) kmax = fmaxf(kmax, kmax_w[w]);
    kmax = sqrtf(kmax);

    const int nsb = (nbw + 1) / 2;
    // A fragment with row 0 all ones (lanes 0-15 hold row 0's k values)
    bf16x8 ones;
#pragma unroll
    for (int i = 0; i < 8; ++i) ones[i] = (__bf16)(col == 0 ? 1.0f : 0.0f);
    // Each wavefront owns a contiguous quarter of the window's query blocks and walks it in
    // passes of QMAX blocks, the last pass with QMAX / 2 (a lone leftover block computes a
    // duplicate that is not stored). Q of the next pass is loaded during the current one.
    const int qend = (wave + 1) * nbw / WAVES;
    auto load_q = [&](int qb0, u16x8 (&qv)[QMAX]) {
#pragma unroll
        for (int j = 0; j < QMAX; ++j) {
            const int qb = min(qb0 + j, qend - 1);
            qv[j] = *reinterpret_cast<const u16x8*>(
                p.QKV + (((tb_base + qb) * 3 + 0) * KSD + frag) * 512 + lane * 8);
        }
    };
    u16x8 qnext[QMAX];
    int qbeg = wave * nbw / WAVES;
    if (qbeg < qend) load_q(qbeg, qnext);
    auto pass = [&](auto qbc, int qb0) {
        constexpr int QB = decltype(qbc)::value;
        u16x8 qv[QB];
#pragma unroll
        for (int j = 0; j < QB; ++j) qv[j] = qnext[j];
        if (qb0 + QB < qend) load_q(qb0 + QB, qnext);   // next pass, in flight
        FT q[QB];
        f32x4 shift[QB];
        float m[QB];
#pragma unroll
        for (int j = 0; j < QB; ++j) {
            float n2 = 0.f;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const float f = (float)__builtin_bit_cast(__bf16, (uint16_t)qv[j][slot0 + i]);
                n2 = fmaf(f, f, n2);
                q[j][i] = __builtin_bit_cast(__bf16, (uint16_t)qv[j][slot0 + i]);
            }
            m[j] = sqrtf(sum4(n2)) * kmax;
            shift[j] = f32x4{-m[j], -m[j], -m[j], -m[j]};
        }

        f32x4 o[QB][RT];
        f32x4 ls[QB];     // row 0 (lanes 0-15, element 0): sum of P over the keys
#pragma unroll
        for (int j = 0; j < QB; ++j) {
            ls[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) o[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

        // K and V^T fragments of superblock sb (two 16-key blocks). Indices up to nsb - 1
        // stay inside the LDS image (a missing last key block reads the start of V^T), so the
        // prefetches below never need a bounds branch; such values are never used.
        auto load_k = [&](int sb, FT (&kf)[2]) {
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) kf[kk] = ld_kfrag<DH>(ks, 2 * sb + kk, lane, slot0);
        };
        auto load_v = [&](int sb, bf16x8 (&vf)[RT]) {
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) vf[rt] = ld_vfrag(vs, DH == 32 ? rt : vhalf, sb, lane);
        };
        // S^T - m of one superblock for every query block
        auto scores = [&](const FT (&kf)[2], f32x4 (&s)[QB][2]) {
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int j = 0; j < QB; ++j) s[j][kk] = Frag<DH>::mma(kf[kk], q[j], shift[j]);
        };
        // P = exp2(S), row sums, and O^T += V^T P^T for one superblock
        auto accumulate = [&](const f32x4 (&s)[QB][2], const bf16x8 (&vf)[RT]) {
            bf16x8 pb[QB];
#pragma unroll
            for (int j = 0; j < QB; ++j) {
                f32x4 pr[2];
#pragma unroll
                for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                    for (int i = 0; i < 4; ++i) pr[kk][i] = exp2_fast(s[j][kk][i]);
                pb[j] = pack_b(pr[0], pr[1]);
                ls[j] = mfma16x16x32(ones, pb[j], ls[j]);
            }
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
#pragma unroll
                for (int j = 0; j < QB; ++j) o[j][rt] = mfma16x16x32(vf[rt], pb[j], o[j][rt]);
        };
        // Every superblock but the last is full. Software pipeline over them, unrolled by two:
        // while the exponentials of sb run, the scores of sb+1 are on the matrix core, K of
        // sb+2 and V of sb+1 are in flight from LDS.
        const int nfull = nsb - 1;
        const int lastsb = nsb - 1;
        FT kA[2], kB[2];
        bf16x8 vA[RT], vB[RT];
        f32x4 sA[QB][2], sB[QB][2];
        load_k(0, kA);
        load_v(0, vA);
        load_k(min(1, lastsb), kB);
        scores(kA, sA);
        int sb = 0;
        for (; sb + 2 <= nfull; sb += 2) {
            scores(kB, sB);                              // sb + 1
            load_k(min(sb + 2, lastsb), kA);
            load_v(sb + 1, vB);
            accumulate(sA, vA);                          // sb
            scores(kA, sA);                              // sb + 2 (unused past nfull)
            load_k(min(sb + 3, lastsb), kB);
            load_v(min(sb + 2, lastsb), vA);
            accumulate(sB, vB);                          // sb + 1
        }
        if (sb < nfull) accumulate(sA, vA);
        {   // last superblock: missing key block and padding keys are -inf
            const int last = nsb - 1;
            f32x4 s[QB][2];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                const int kb = 2 * last + kk;
                if (kb < nbw) {
                    const FT a = ld_kfrag<DH>(ks, kb, lane, slot0);
#pragma unroll
                    for (int j = 0; j < QB; ++j) s[j][kk] = Frag<DH>::mma(a, q[j], shift[j]);
                } else {
#pragma unroll
                    for (int j = 0; j < QB; ++j) s[j][kk] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (kb * 16 + 4 * g + i >= N)
#pragma unroll
                        for (int j = 0; j < QB; ++j) s[j][kk][i] = -INFINITY;
            }
            bf16x8 vl[RT];
            load_v(last, vl);
            accumulate(s, vl);
        }

#pragma unroll
        for (int j = 0; j < QB; ++j) {
            const int qb = qb0 + j;
            float lt = __shfl(ls[j][0], col);   // row 0 of the sums lives in lane col
            // underflowed row sums: redo this block with a running maximum (wave-uniform)
            if (__builtin_amdgcn_ballot_w64(lt < 1e-30f) != 0) {
                float mm = -INFINITY, ll = 0.f;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) o[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
                const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
                for (int sb = 0; sb < nsb; ++sb) {
                    f32x4 s2[2];
                    for (int kk = 0; kk < 2; ++kk) {
                        const int kb = 2 * sb + kk;
                        if (kb < nbw) s2[kk] = Frag<DH>::mma(ld_kfrag<DH>(ks, kb, lane, slot0), q[j], zero);
                        else s2[kk] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
                        for (int i = 0; i < 4; ++i)
                            if (kb * 16 + 4 * g + i >= N) s2[kk][i] = -INFINITY;
                    }
                    float mx = fmaxf(fmaxf(fmaxf(s2[0][0], s2[0][1]), fmaxf(s2[0][2], s2[0][3])),
                                     fmaxf(fmaxf(s2[1][0], s2[1][1]), fmaxf(s2[1][2], s2[1][3])));
                    mx = fmaxf(mx, __shfl_xor(mx, 16));
                    mx = fmaxf(mx, __shfl_xor(mx, 32));
                    const float mnew = fmaxf(mm, mx);
                    const float alpha = exp2_fast(mm - mnew);
                    f32x4 pr[2];
                    float ls = 0.f;
                    for (int kk = 0; kk < 2; ++kk)
                        for (int i = 0; i < 4; ++i) {
                            pr[kk][i] = exp2_fast(s2[kk][i] - mnew);
                            ls += pr[kk][i];
                        }
                    ll = ll * alpha + ls;
                    mm = mnew;
                    const bf16x8 pb2 = pack_b(pr[0], pr[1]);
                    for (int rt = 0; rt < RT; ++rt)
                        o[j][rt] = mfma16x16x32(ld_vfrag(vs, DH == 32 ? rt : vhalf, sb, lane), pb2, o[j][rt] * alpha);
                }
                lt = sum4(ll);
            }
            if (qb >= qend) continue;
            const float inv = 1.0f / lt;
            uint16_t* dst = p.Y + ((tb_base + qb) * KSD + frag) * 512 + lane * 8;
            if constexpr (DH == 32) {
                const bf16x8 out = pack_b(o[j][0] * inv, o[j][RT - 1] * inv);
                *reinterpret_cast<u16x8*>(dst) = __builtin_bit_cast(u16x8, out);
            } else {
                u16x4 out;
#pragma unroll
                for (int i = 0; i < 4; ++i) out[i] = __builtin_bit_cast(uint16_t, (__bf16)(o[j][0][i] * inv));
                *reinterpret_cast<u16x4*>(dst + slot0) = out;
            }
        }
    };
    int qb = qbeg;
    for (; qend - qb >= QMAX - 1; qb += QMAX) pass(std::integral_constant<int, QMAX>{}, qb);
    if (qb < qend) pass(std::integral_constant<int, QMAX / 2>{}, qb);
}

}  // namespace

size_t attn_smem_bytes(int dh, int Npad, int nbw) {
    (void)dh;
    (void)Npad;
    return (size_t)(2 * nbw + 1) * 1024;   // K [nbw] and V [nbw + 1] fragments of 1 KB
}

template <int DH, int WAVES>
hipError_t launch_shape(const AttnParams& p, int nwin, hipStream_t s) {
    const size_t smem = attn_smem_bytes(DH, p.Npad, p.nbw);
    hipError_t e = hipFuncSetAttribute((const void*)attn_kernel<DH, WAVES>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    attn_kernel<DH, WAVES><<<dim3((unsigned)nwin * p.H), dim3(WAVES * 64), smem, s>>>(p);
    return hipGetLastError();
}

template <int DH>
hipError_t launch_dh(const AttnParams& p, int nwin, hipStream_t s) {
    // wavefronts per (window, head): enough for a pass of QMAX query blocks each, at most
    // four, so small windows run as many small workgroups rather than idle wavefronts
    if (p.nbw <= QMAX) return launch_shape<DH, 1>(p, nwin, s);
    if (p.nbw <= 2 * QMAX) return launch_shape<DH, 2>(p, nwin, s);
    return launch_shape<DH, 4>(p, nwin, s);
}

hipError_t launch_attn(int dh, const AttnParams& p, int nwin, hipStream_t s) {
    if (nwin <= 0) return hipSuccess;
    if (dh == 32) return launch_dh<32>(p, nwin, s);
    if (dh == 16) return launch_dh<16>(p, nwin, s);
    return hipErrorInvalidValue;
}
