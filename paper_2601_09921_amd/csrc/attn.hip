// Multi-head self-attention across the stabilizer tokens of each window (App. A.2; the
// model table's Multi-Head Attention), bf16 MFMA with fp32 softmax statistics.
//
// One workgroup per (window, head). K_h (as MFMA A fragments) and V_h^T are staged in LDS
// once; each wavefront then takes 16-query blocks and streams the keys in steps of 32:
//   S^T = K Q^T             (16 keys x 16 queries per MFMA, lanes hold queries)
//   online softmax           (running max and sum per query, exp2 with log2(e)/sqrt(dh))
//   O^T += V^T P^T           (P^T is the S^T accumulator rounded to bf16, no shuffle)
// Padding keys (index >= N) get probability 0. The output is written as the B fragments
// the out-projection consumes.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int WAVES = 4;

__host__ __device__ inline int vt_stride(int Npad) { return ((Npad + 31) & ~31) + 8; }   // + 8: spread banks

template <int DH>
__global__ __launch_bounds__(WAVES * 64) void attn_kernel(AttnParams p) {
    constexpr int RT = DH / 16;                 // 16-row tiles of O^T
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    const int win = blockIdx.x / p.H, h = blockIdx.x % p.H;
    const int nbw = p.nbw;
    const int KSD = p.H * DH / 32;              // k-steps of D (fragments per Q/K/V)
    const int64_t tb_base = (int64_t)win * nbw;
    const int vts = vt_stride(p.Npad);

    extern __shared__ __align__(16) unsigned char smem[];
    // K fragments: DH 32 -> 8 bf16 per lane, DH 16 -> 4 bf16 per lane
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem);
    uint16_t* vt = ks + (size_t)nbw * 64 * (DH == 32 ? 8 : 4);

    // fragment and slot range of head h inside a Q/K/V fragment
    const int frag = DH == 32 ? h : h / 2;
    const int slot0 = DH == 32 ? 0 : (h % 2) * 4;

    for (int kb = wave; kb < nbw; kb += WAVES) {
        const uint16_t* src = p.QKV + (((tb_base + kb) * 3 + 1) * KSD + frag) * 512 + lane * 8;
        const u16x8 kv = *reinterpret_cast<const u16x8*>(src);
        if (DH == 32) {
            *reinterpret_cast<u16x8*>(ks + (kb * 64 + lane) * 8) = kv;
        } else {
            u16x4 k4;
            for (int i = 0; i < 4; ++i) k4[i] = kv[slot0 + i];
            *reinterpret_cast<u16x4*>(ks + (kb * 64 + lane) * 4) = k4;
        }
        const uint16_t* vsrc = p.QKV + (((tb_base + kb) * 3 + 2) * KSD + frag) * 512 + lane * 8;
        const u16x8 vv = *reinterpret_cast<const u16x8*>(vsrc);
        const int key = kb * 16 + col;
        if (DH == 32) {
            for (int i = 0; i < 8; ++i) vt[kslot(g, i) * vts + key] = vv[i];
        } else {
            for (int i = 0; i < 4; ++i) vt[(4 * g + i) * vts + key] = vv[slot0 + i];
        }
    }
    // zero the key tail [Npad, 32*ceil(Npad/32)) so P = 0 never meets garbage
    const int kpad = (p.Npad + 31) & ~31;
    for (int idx = threadIdx.x; idx < DH * (kpad - p.Npad); idx += blockDim.x) {
        const int r = idx / (kpad - p.Npad), k = p.Npad + idx % (kpad - p.Npad);
        vt[r * vts + k] = 0;
    }
    __syncthreads();

    const float c = p.scale_log2;
    const int nsb = (nbw + 1) / 2;
    for (int qb = wave; qb < nbw; qb += WAVES) {
        const uint16_t* qsrc = p.QKV + (((tb_base + qb) * 3 + 0) * KSD + frag) * 512 + lane * 8;
        const u16x8 qv = *reinterpret_cast<const u16x8*>(qsrc);
        bf16x8 q8 = __builtin_bit_cast(bf16x8, qv);
        bf16x4 q4;
        for (int i = 0; i < 4; ++i) q4[i] = q8[slot0 + i];

        f32x4 o[RT];
        for (int rt = 0; rt < RT; ++rt) o[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
        float m = -INFINITY, l = 0.f;

        for (int sb = 0; sb < nsb; ++sb) {
            f32x4 s[2];
            for (int j = 0; j < 2; ++j) {
                const int kb = 2 * sb + j;
                if (kb < nbw) {
                    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
                    if (DH == 32) {
                        const bf16x8 a = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(ks + (kb * 64 + lane) * 8));
                        s[j] = mfma16x16x32(a, q8, zero);
                    } else {
                        const bf16x4 a = __builtin_bit_cast(bf16x4, *reinterpret_cast<const u16x4*>(ks + (kb * 64 + lane) * 4));
                        s[j] = mfma16x16x16(a, q4, zero);
                    }
                    for (int i = 0; i < 4; ++i)
                        if (kb * 16 + 4 * g + i >= p.N) s[j][i] = -INFINITY;
                } else {
                    s[j] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
                }
            }
            float mx = fmaxf(fmaxf(fmaxf(s[0][0], s[0][1]), fmaxf(s[0][2], s[0][3])),
                             fmaxf(fmaxf(s[1][0], s[1][1]), fmaxf(s[1][2], s[1][3])));
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mnew = fmaxf(m, mx);
            const float alpha = exp2f((m - mnew) * c);
            const float mc = mnew * c;
            f32x4 pr[2];
            float ls = 0.f;
            for (int j = 0; j < 2; ++j)
                for (int i = 0; i < 4; ++i) {
                    pr[j][i] = exp2f(s[j][i] * c - mc);
                    ls += pr[j][i];
                }
            l = l * alpha + ls;
            m = mnew;
            const bf16x8 pb = pack_b(pr[0], pr[1]);
            for (int rt = 0; rt < RT; ++rt) {
                const uint16_t* row = vt + (rt * 16 + col) * vts + 32 * sb + 4 * g;
                u16x8 v;
                const u16x4 lo = *reinterpret_cast<const u16x4*>(row);
                const u16x4 hi = *reinterpret_cast<const u16x4*>(row + 16);
                for (int i = 0; i < 4; ++i) {
                    v[i] = lo[i];
                    v[4 + i] = hi[i];
                }
                o[rt] = o[rt] * alpha;
                o[rt] = mfma16x16x32(__builtin_bit_cast(bf16x8, v), pb, o[rt]);
            }
        }
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        const float inv = 1.0f / l;
        uint16_t* dst = p.Y + ((tb_base + qb) * KSD + frag) * 512 + lane * 8;
        if constexpr (DH == 32) {
            const bf16x8 out = pack_b(o[0] * inv, o[RT - 1] * inv);
            *reinterpret_cast<u16x8*>(dst) = __builtin_bit_cast(u16x8, out);
        } else {
            u16x4 out;
            for (int i = 0; i < 4; ++i) out[i] = __builtin_bit_cast(uint16_t, (__bf16)(o[0][i] * inv));
            *reinterpret_cast<u16x4*>(dst + slot0) = out;
        }
    }
}

}  // namespace

size_t attn_smem_bytes(int dh, int Npad, int nbw) {
    return (size_t)nbw * 64 * (dh == 32 ? 8 : 4) * 2 + (size_t)dh * vt_stride(Npad) * 2;
}

hipError_t launch_attn(int dh, const AttnParams& p, int nwin, hipStream_t s) {
    if (nwin <= 0) return hipSuccess;
    const size_t smem = attn_smem_bytes(dh, p.Npad, p.nbw);
    const dim3 grid((unsigned)nwin * p.H), block(WAVES * 64);
    if (dh == 32) {
        hipError_t e = hipFuncSetAttribute((const void*)attn_kernel<32>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return e;
        attn_kernel<32><<<grid, block, smem, s>>>(p);
    } else if (dh == 16) {
        hipError_t e = hipFuncSetAttribute((const void*)attn_kernel<16>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return e;
        attn_kernel<16><<<grid, block, smem, s>>>(p);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}
