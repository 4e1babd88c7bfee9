// Multi-head self-attention across the stabilizer tokens of each window (App. A.2; the
// model table's Multi-Head Attention), bf16 MFMA with fp32 softmax statistics.
//
// The unit of work is one (window, head): K_h and V_h are copied to LDS by direct
// global->LDS loads of the fragments the Q/K/V projection wrote (K as B fragments of K^T,
// which serve as A fragments of K; V as 16x16 tiles with tokens as rows, whose per-lane
// halves of two key blocks form an A fragment of V^T); the wavefronts then split the
// 16-query blocks and stream the keys in steps of 32:
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
//
// One workgroup of 1, 2 or 4 wavefronts (by window size) per item, two workgroups per CU:
// while one copies its K/V, the other keeps the SIMDs busy.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int QMAX = 4;               // query blocks per wavefront pass, at most
constexpr int KMAX_UNROLL = 8;        // key blocks per step of the max |k| scan

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

// Sizes shared by every item of a launch.
struct AttnShape {
    int N, nbw, KSD;   // real tokens, 16-token blocks, Q/K/V fragments per token block
};

// One (window, head) item: its K/V in LDS, its Q, K and Y in HBM, and max |k|.
struct AttnItem {
    const uint16_t* ks;   // LDS [nbw][512] K fragments
    const uint16_t* vs;   // LDS [nbw + 1][512] V tiles (+ a zero block when nbw is odd)
    const uint16_t* q0;   // Q fragment of token block 0; block stride 3 KSD fragments
    const uint16_t* k0;   // K fragment of token block 0 (V follows at + KSD fragments)
    uint16_t* y0;         // Y fragment of token block 0; block stride KSD fragments
    int slot0, vhalf;     // this head's slots inside a fragment (dh = 16 packs two heads)
    float kmax;
};

template <int DH>
PWD_DEV AttnItem make_item(const AttnParams& p, const AttnShape& sh, int item) {
    const int win = item / p.H, h = item % p.H;
    const int frag = DH == 32 ? h : h / 2;
    const int64_t tb_base = (int64_t)win * sh.nbw;
    AttnItem it;
    it.ks = it.vs = nullptr;
    it.q0 = p.QKV + (tb_base * 3 * sh.KSD + frag) * 512;
    it.k0 = it.q0 + (size_t)sh.KSD * 512;
    it.y0 = p.Y + (tb_base * sh.KSD + frag) * 512;
    it.slot0 = DH == 32 ? 0 : (h % 2) * 4;
    it.vhalf = DH == 32 ? 0 : h % 2;
    it.kmax = 0.f;
    return it;
}

// Q of the QMAX blocks from qb0 (indices past qend - 1 repeat the last block).
PWD_DEV void load_q(const AttnShape& sh, const uint16_t* q0, int qb0, int qend, int lane, u16x8 (&qv)[QMAX]) {
#pragma unroll
    for (int j = 0; j < QMAX; ++j) {
        const int qb = min(qb0 + j, qend - 1);
        qv[j] = *reinterpret_cast<const u16x8*>(q0 + (size_t)qb * 3 * sh.KSD * 512 + lane * 8);
    }
}

// Direct copies of the K and V fragments of key blocks kb0, kb0 + stride, ... into LDS.
PWD_DEV void stage_kv(const AttnShape& sh, const uint16_t* k0, uint16_t* ks, uint16_t* vs, int kb0, int stride,
                      int lane) {
    for (int kb = kb0; kb < sh.nbw; kb += stride) {
        const uint16_t* src = k0 + (size_t)kb * 3 * sh.KSD * 512;
        lds_load_1k(uniform_ptr(src), lds_addr(ks + kb * 512), lane);
        lds_load_1k(uniform_ptr(src + (size_t)sh.KSD * 512), lds_addr(vs + kb * 512), lane);
    }
}

// max |k|^2 over the real keys of blocks kb0, kb0 + stride, ..., reduced over the wavefront;
// KMAX_UNROLL blocks at a time so their LDS reads and cross-lane sums are in flight together.
// Blocks past the last are skipped (the tests are wavefront-uniform).
template <int DH>
PWD_DEV float kmax2_blocks(const AttnShape& sh, const uint16_t* ks, int slot0, int kb0, int stride, int lane) {
    constexpr int NV = DH == 32 ? 8 : 4;
    const int col = lane & 15;
    float kmax2 = 0.f;
    for (int kbs = kb0; kbs < sh.nbw; kbs += KMAX_UNROLL * stride) {
        float n2[KMAX_UNROLL];
#pragma unroll
        for (int u = 0; u < KMAX_UNROLL; ++u) {
            const int kb = kbs + u * stride;
            n2[u] = 0.f;
            if (kb < sh.nbw) {
                const u16x8 kv = *reinterpret_cast<const u16x8*>(ks + (kb * 64 + lane) * 8);
#pragma unroll
                for (int i = 0; i < NV; ++i) {
                    const float f = (float)__builtin_bit_cast(__bf16, (uint16_t)kv[slot0 + i]);
                    n2[u] = fmaf(f, f, n2[u]);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < KMAX_UNROLL; ++u)
            if (kbs + u * stride < sh.nbw) n2[u] += __shfl_xor(n2[u], 16);
#pragma unroll
        for (int u = 0; u < KMAX_UNROLL; ++u)
            if (kbs + u * stride < sh.nbw) n2[u] += __shfl_xor(n2[u], 32);
#pragma unroll
        for (int u = 0; u < KMAX_UNROLL; ++u) {
            const int kb = kbs + u * stride;
            if (kb < sh.nbw && kb * 16 + col < sh.N) kmax2 = fmaxf(kmax2, n2[u]);
        }
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) kmax2 = fmaxf(kmax2, __shfl_xor(kmax2, off));
    return kmax2;
}

// Scheduling request for one iteration of the key loop (two superblocks, 20 QB MFMAs): each
// MFMA followed by three VALU or transcendental instructions, so the exponentials and packs
// issue while the matrix core runs instead of in separate bursts (measured: 3 per MFMA beats
// 2 and 4).
template <int NMFMA>
PWD_DEV void interleave_mfma_valu() {
#pragma unroll
    for (int i = 0; i < NMFMA; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
        __builtin_amdgcn_sched_group_barrier(0x402, 3, 0);   // VALU or TRANS
    }
}

// One pass of a wavefront: query blocks qb0 .. qb0 + QB - 1 (those >= qend are computed
// from a repeated block and not stored) against every key of the item.
template <int DH, int QB>
PWD_DEV void attn_pass(const AttnShape& sh, const AttnItem& it, int qb0, int qend, const u16x8 (&qv)[QMAX],
                       const bf16x8& ones, int lane) {
    using FT = typename Frag<DH>::T;
    constexpr int RT = DH / 16;                 // 16-row tiles of O^T
    constexpr int NV = DH == 32 ? 8 : 4;        // Q/K values per lane
    const int g = lane >> 4, col = lane & 15;
    const int nbw = sh.nbw, N = sh.N, slot0 = it.slot0;
    const int nsb = (nbw + 1) / 2;
    const uint16_t* ks = it.ks;
    const uint16_t* vs = it.vs;

    FT q[QB];
    f32x4 shift[QB];
#pragma unroll
    for (int j = 0; j < QB; ++j) {
        float n2 = 0.f;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const float f = (float)__builtin_bit_cast(__bf16, (uint16_t)qv[j][slot0 + i]);
            n2 = fmaf(f, f, n2);
            q[j][i] = __builtin_bit_cast(__bf16, (uint16_t)qv[j][slot0 + i]);
        }
        const float m = sqrtf(sum4(n2)) * it.kmax;
        shift[j] = f32x4{-m, -m, -m, -m};
    }

    f32x4 o[QB][RT];
    f32x4 ls[QB];     // row 0 (lanes 0-15, element 0): sum of P over the keys
#pragma unroll
    for (int j = 0; j < QB; ++j) {
        ls[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) o[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // K and V^T fragments of superblock sb (two 16-key blocks). Indices up to nsb - 1 stay
    // inside the LDS image (a missing last key block reads the start of V^T), so the
    // prefetches below never need a bounds branch; such values are never used.
    auto load_k = [&](int sb, FT (&kf)[2]) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) kf[kk] = ld_kfrag<DH>(ks, 2 * sb + kk, lane, slot0);
    };
    auto load_v = [&](int sb, bf16x8 (&vf)[RT]) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) vf[rt] = ld_vfrag(vs, DH == 32 ? rt : it.vhalf, sb, lane);
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
        interleave_mfma_valu<10 * QB>();
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
            if (kb < nbw && (kb + 1) * 16 > N)   // a real block with padding keys (uniform test)
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
                float lsum = 0.f;
                for (int kk = 0; kk < 2; ++kk)
                    for (int i = 0; i < 4; ++i) {
                        pr[kk][i] = exp2_fast(s2[kk][i] - mnew);
                        lsum += pr[kk][i];
                    }
                ll = ll * alpha + lsum;
                mm = mnew;
                const bf16x8 pb2 = pack_b(pr[0], pr[1]);
                for (int rt = 0; rt < RT; ++rt)
                    o[j][rt] = mfma16x16x32(ld_vfrag(vs, DH == 32 ? rt : it.vhalf, sb, lane), pb2, o[j][rt] * alpha);
            }
            lt = sum4(ll);
        }
        if (qb >= qend) continue;
        const float inv = 1.0f / lt;
        uint16_t* dst = it.y0 + (size_t)qb * sh.KSD * 512 + lane * 8;
        if constexpr (DH == 32) {
            const bf16x8 out = pack_b(o[j][0] * inv, o[j][RT - 1] * inv);
            *reinterpret_cast<u16x8*>(dst) = __builtin_bit_cast(u16x8, out);
        } else {
            u16x4 out;
#pragma unroll
            for (int i = 0; i < 4; ++i) out[i] = __builtin_bit_cast(uint16_t, (__bf16)(o[j][0][i] * inv));
            *reinterpret_cast<u16x4*>(dst + it.slot0) = out;
        }
    }
}

// A fragment with row 0 all ones (lanes 0-15 hold row 0's k values)
PWD_DEV bf16x8 ones_row(int lane) {
    bf16x8 ones;
#pragma unroll
    for (int i = 0; i < 8; ++i) ones[i] = (__bf16)((lane & 15) == 0 ? 1.0f : 0.0f);
    return ones;
}

// Passes of QMAX, 2 and 1 blocks over this wavefront's query blocks [qbeg, qend). qnext
// holds Q of the first pass on entry; each pass first starts the Q load of the pass after it.
template <int DH>
PWD_DEV void attn_passes(const AttnShape& sh, const AttnItem& it, int qbeg, int qend, u16x8 (&qnext)[QMAX],
                         const bf16x8& ones, int lane) {
    auto prefetch = [&](int qb_after) {
        if (qb_after < qend) load_q(sh, it.q0, qb_after, qend, lane, qnext);
    };
    int qb = qbeg;
    while (qend - qb >= QMAX) {
        u16x8 qv[QMAX];
#pragma unroll
        for (int j = 0; j < QMAX; ++j) qv[j] = qnext[j];
        prefetch(qb + QMAX);
        attn_pass<DH, QMAX>(sh, it, qb, qend, qv, ones, lane);
        qb += QMAX;
    }
    if (qend - qb >= 2) {
        u16x8 qv[QMAX];
#pragma unroll
        for (int j = 0; j < QMAX; ++j) qv[j] = qnext[j];
        prefetch(qb + 2);
        attn_pass<DH, 2>(sh, it, qb, qend, qv, ones, lane);
        qb += 2;
    }
    if (qend - qb == 1) {
        u16x8 qv[QMAX];
#pragma unroll
        for (int j = 0; j < QMAX; ++j) qv[j] = qnext[j];
        prefetch(qb + 1);
        attn_pass<DH, 1>(sh, it, qb, qend, qv, ones, lane);
    }
}

// One workgroup per (window, head); K/V stay in LDS for the whole item.
template <int DH, int WAVES>
__global__ __launch_bounds__(WAVES * 64, 2) void attn_kernel(AttnParams p) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const AttnShape sh{p.N, p.nbw, p.H * DH / 32};
    const int nbw = sh.nbw;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem);   // [nbw][512]: K fragments
    uint16_t* vs = ks + (size_t)nbw * 512;               // [nbw + 1][512]: V tiles, + a zero block
    __shared__ float kmax_w[WAVES];
    AttnItem it = make_item<DH>(p, sh, blockIdx.x);
    it.ks = ks;
    it.vs = vs;

    // Each wavefront owns a contiguous share of the query blocks; Q of its first pass is
    // loaded before the K/V staging, so its latency overlaps the staging.
    const int qbeg = wave * nbw / WAVES, qend = (wave + 1) * nbw / WAVES;
    u16x8 qnext[QMAX];
    if (qbeg < qend) load_q(sh, it.q0, qbeg, qend, lane, qnext);

    // stage K and V; an odd key-block count gets a zero V block so the last superblock's
    // missing keys meet P = 0 and V = 0
    stage_kv(sh, it.k0, ks, vs, wave, WAVES, lane);
    if (nbw & 1)
        for (int i = threadIdx.x; i < 256; i += blockDim.x) reinterpret_cast<uint32_t*>(vs + nbw * 512)[i] = 0u;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    const float kw = kmax2_blocks<DH>(sh, ks, it.slot0, wave, WAVES, lane);
    if (lane == 0) kmax_w[wave] = kw;
    __syncthreads();
    float kmax2 = 0.f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) kmax2 = fmaxf(kmax2, kmax_w[w]);
    it.kmax = sqrtf(kmax2);
    if (qbeg < qend) attn_passes<DH>(sh, it, qbeg, qend, qnext, ones_row(lane), lane);
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

}  // namespace

size_t attn_smem_bytes(int dh, int Npad, int nbw) {
    (void)dh;
    (void)Npad;
    return (size_t)(2 * nbw + 1) * 1024;   // K [nbw] and V [nbw + 1] fragments of 1 KB
}

hipError_t launch_attn(int dh, const AttnParams& p, int nwin, hipStream_t s) {
    if (nwin <= 0) return hipSuccess;
    if (dh == 32) return launch_dh<32>(p, nwin, s);
    if (dh == 16) return launch_dh<16>(p, nwin, s);
    return hipErrorInvalidValue;
}
