// Multi-head self-attention across the stabilizer tokens of each window (App. A.2; the
// model table's Multi-Head Attention), bf16 MFMA with fp32 softmax statistics.
//
// The unit of work is one (window, head): K_h and V_h are copied to LDS by direct
// global->LDS loads of the fragments the Q/K/V projection wrote (K as B fragments of K^T,
// which serve as A fragments of K; V as 16x16 tiles with tokens as rows, whose per-lane
// halves of two key blocks form an A fragment of V^T); the wavefronts then split the
// 16-query blocks and stream the keys in steps of 32:
//   S^T = K Q'^T          (16 keys x 16 queries per MFMA, lanes hold queries)
//   P^T = exp2(S^T)       (P^T is the S^T accumulator rounded to bf16, no shuffle)
//   O^T += V^T P^T,  l += 1^T P^T
// Q' = Q log2(e)/sqrt(dh) comes pre-scaled from the Q/K/V projection, so S is in log2 units.
// Softmax is shift-invariant, so the scores are exponentiated as they are: with fp32
// exponentials, bf16 probabilities and fp32 sums this is the exact softmax (up to rounding)
// whenever every probability and partial sum stays in the normal fp32 range, which a score
// range of about +-100 log2 units guarantees. A query block whose row sum or output leaves
// that range (inf, NaN, or a sum below 1e-30) is recomputed with the running-maximum form,
// so no input is out of reach; the common case spends no VALU work on a shift. Padding keys
// (index >= N) get probability 0. The row sums l come from the matrix core too: an A
// fragment whose row 0 is all ones turns P^T into its column sums, so numerator and
// denominator use the same bf16 probabilities and the VALU is left to the exponentials. The
// output is written as the B fragments the out-projection consumes.
//
// One workgroup of 1, 2, 4 or 8 wavefronts per item, as many workgroups per CU as their K/V
// tiles fit in LDS (two wavefronts per SIMD in all): while some copy their K/V, the others
// keep the SIMDs busy.
#include "common.h"
#include "kernels.h"

namespace {

#ifndef ATTN_WIDE
#define ATTN_WIDE 1
#endif

PWD_DEV float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Head sizes: a Q/K/V fragment holds 32 features of 16 tokens, so a head of 64 spans NF = 2
// fragments per token block (its scores take two 32-deep k-steps), a head of 32 one, and a
// head of 16 half of one (slot0 selects its four values in each lane).
template <int DH>
struct Frag;
template <>
struct Frag<64> {
    using T = bf16x8;
    static constexpr int NF = 2, NV = 8, QMAX = 2;
    static __device__ __forceinline__ f32x4 mma(T a, T b, f32x4 c) { return mfma16x16x32(a, b, c); }
};
template <>
struct Frag<32> {
    using T = bf16x8;
    static constexpr int NF = 1, NV = 8, QMAX = 4;
    static __device__ __forceinline__ f32x4 mma(T a, T b, f32x4 c) { return mfma16x16x32(a, b, c); }
};
template <>
struct Frag<16> {
    using T = bf16x4;
    static constexpr int NF = 1, NV = 4, QMAX = 4;
    static __device__ __forceinline__ f32x4 mma(T a, T b, f32x4 c) { return mfma16x16x16(a, b, c); }
};

// K fragment f of key block kb (LDS holds whole 1 KB fragments, NF per key block).
template <int DH>
PWD_DEV typename Frag<DH>::T ld_kfrag(const uint16_t* ks, int kb, int f, int lane, int slot0) {
    const uint16_t* src = ks + ((kb * Frag<DH>::NF + f) * 64 + lane) * 8;
    if constexpr (DH == 16)
        return __builtin_bit_cast(bf16x4, *reinterpret_cast<const u16x4*>(src + slot0));
    else
        return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(src));
}

// V^T A fragment of the 32 keys of superblock sb for head features 16 t .. 16 t + 15 (tile t
// = half `half` of V fragment f): this lane's four keys of key block 2 sb (k slots 0-3) and of
// key block 2 sb + 1 (k slots 4-7), i.e. the lane's 8 bytes of that tile in both blocks.
template <int NF>
PWD_DEV bf16x8 ld_vfrag(const uint16_t* vs, int f, int half, int sb, int lane) {
    const uint16_t* t = vs + ((2 * sb) * NF + f) * 512 + half * 256 + lane * 4;
    const u16x4 lo = *reinterpret_cast<const u16x4*>(t);
    const u16x4 hi = *reinterpret_cast<const u16x4*>(t + NF * 512);
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

// One (window, head) item: its K/V in LDS, its Q, K and Y in HBM.
struct AttnItem {
    const uint16_t* ks;   // LDS [nbw][NF][512] K fragments
    const uint16_t* vs;   // LDS [nbw + 1][NF][512] V tiles (+ a zero block when nbw is odd)
    const uint16_t* q0;   // first Q fragment of token block 0; block stride 3 KSD fragments
    const uint16_t* k0;   // first K fragment of token block 0 (V follows at + KSD fragments)
    uint16_t* y0;         // first Y fragment of token block 0; block stride KSD fragments
    int slot0, vhalf;     // this head's slots inside a fragment (dh = 16 packs two heads)
};

template <int DH>
PWD_DEV AttnItem make_item(const AttnParams& p, const AttnShape& sh, int item) {
    const int win = item / p.H, h = item % p.H;
    const int frag = DH == 64 ? 2 * h : DH == 32 ? h : h / 2;
    const int64_t tb_base = (int64_t)win * sh.nbw;
    AttnItem it;
    it.ks = it.vs = nullptr;
    it.q0 = p.QKV + (tb_base * 3 * sh.KSD + frag) * 512;
    it.k0 = it.q0 + (size_t)sh.KSD * 512;
    it.y0 = p.Y + (tb_base * sh.KSD + frag) * 512;
    it.slot0 = DH == 16 ? (h % 2) * 4 : 0;
    it.vhalf = DH == 16 ? h % 2 : 0;
    return it;
}

// Q of the QM blocks from qb0 (indices past qend - 1 repeat the last block), NF fragments each.
template <int NF, int QM>
PWD_DEV void load_q(const AttnShape& sh, const uint16_t* q0, int qb0, int qend, int lane, u16x8 (&qv)[QM][NF]) {
#pragma unroll
    for (int j = 0; j < QM; ++j) {
        const int qb = min(qb0 + j, qend - 1);
#pragma unroll
        for (int f = 0; f < NF; ++f)
            qv[j][f] = *reinterpret_cast<const u16x8*>(q0 + ((size_t)qb * 3 * sh.KSD + f) * 512 + lane * 8);
    }
}

// Direct copies of the K and V fragments of key blocks kb0, kb0 + stride, ... into LDS.
template <int NF>
PWD_DEV void stage_kv(const AttnShape& sh, const uint16_t* k0, uint16_t* ks, uint16_t* vs, int kb0, int stride,
                      int lane) {
    for (int kb = kb0; kb < sh.nbw; kb += stride)
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const uint16_t* src = k0 + ((size_t)kb * 3 * sh.KSD + f) * 512;
            lds_load_1k(uniform_ptr(src), lds_addr(ks + (kb * NF + f) * 512), lane);
            lds_load_1k(uniform_ptr(src + (size_t)sh.KSD * 512), lds_addr(vs + (kb * NF + f) * 512), lane);
        }
}

// Scheduling request for one iteration of the key loop (two superblocks, NMFMA MFMAs): each
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
PWD_DEV void attn_pass(const AttnShape& sh, const AttnItem& it, int qb0, int qend,
                       const u16x8 (&qv)[Frag<DH>::QMAX][Frag<DH>::NF], const bf16x8& ones, int lane) {
    using FT = typename Frag<DH>::T;
    constexpr int NF = Frag<DH>::NF, NV = Frag<DH>::NV;
    constexpr int RT = DH / 16;                 // 16-row tiles of O^T
    const int g = lane >> 4, col = lane & 15;
    const int nbw = sh.nbw, N = sh.N, slot0 = it.slot0;
    const int nsb = (nbw + 1) / 2;
    const uint16_t* ks = it.ks;
    const uint16_t* vs = it.vs;

    FT q[QB][NF];
#pragma unroll
    for (int j = 0; j < QB; ++j)
#pragma unroll
        for (int f = 0; f < NF; ++f)
#pragma unroll
            for (int i = 0; i < NV; ++i) q[j][f][i] = __builtin_bit_cast(__bf16, (uint16_t)qv[j][f][slot0 + i]);
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};

    f32x4 o[QB][RT];
    f32x4 ls[QB];     // row 0 (lanes 0-15, element 0): sum of P over the keys
#pragma unroll
    for (int j = 0; j < QB; ++j) {
        ls[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) o[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // V^T tile rt: half rt % 2 of fragment rt / 2 (dh = 16: this head's half of fragment 0)
    auto vtile = [&](int rt, int sb) { return ld_vfrag<NF>(vs, DH == 16 ? 0 : rt / 2, DH == 16 ? it.vhalf : rt % 2, sb, lane); };
    // S^T of key block kb for query block j: NF k-steps over the head's features
    auto score = [&](const FT (&kf)[NF], int j, f32x4 init) {
        f32x4 acc = Frag<DH>::mma(kf[0], q[j][0], init);
#pragma unroll
        for (int f = 1; f < NF; ++f) acc = Frag<DH>::mma(kf[f], q[j][f], acc);
        return acc;
    };
    // K and V^T fragments of superblock sb (two 16-key blocks). Indices up to nsb - 1 stay
    // inside the LDS image (a missing last key block reads the start of V^T), so the
    // prefetches below never need a bounds branch; such values are never used.
    auto load_k = [&](int sb, FT (&kf)[2][NF]) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int f = 0; f < NF; ++f) kf[kk][f] = ld_kfrag<DH>(ks, 2 * sb + kk, f, lane, slot0);
    };
    auto load_v = [&](int sb, bf16x8 (&vf)[RT]) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) vf[rt] = vtile(rt, sb);
    };
    // S^T of one superblock for every query block
    auto scores = [&](const FT (&kf)[2][NF], f32x4 (&s)[QB][2]) {
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int j = 0; j < QB; ++j) s[j][kk] = score(kf[kk], j, zero);
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
    FT kA[2][NF], kB[2][NF];
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
        interleave_mfma_valu<2 * QB * (2 * NF + 1 + RT)>();
    }
    if (sb < nfull) accumulate(sA, vA);
    {   // last superblock: missing key block and padding keys are -inf
        const int last = nsb - 1;
        f32x4 s[QB][2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            const int kb = 2 * last + kk;
            if (kb < nbw) {
                FT a[NF];
#pragma unroll
                for (int f = 0; f < NF; ++f) a[f] = ld_kfrag<DH>(ks, kb, f, lane, slot0);
#pragma unroll
                for (int j = 0; j < QB; ++j) s[j][kk] = score(a, j, zero);
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
        // x * 0 is 0 for finite x and NaN for inf or NaN: chk is lt unless an output is not finite
        float chk = lt;
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int i = 0; i < 4; ++i) chk = fmaf(o[j][rt][i], 0.f, chk);
        // a row sum below 1e-30, above 2^126, or a non-finite output: redo this block with a
        // running maximum (wave-uniform)
        if (__builtin_amdgcn_ballot_w64(!(chk >= 1e-30f && chk <= 0x1p126f)) != 0) {
            float mm = -INFINITY, ll = 0.f;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) o[j][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
            for (int sb = 0; sb < nsb; ++sb) {
                f32x4 s2[2];
                for (int kk = 0; kk < 2; ++kk) {
                    const int kb = 2 * sb + kk;
                    if (kb < nbw) {
                        FT a[NF];
                        for (int f = 0; f < NF; ++f) a[f] = ld_kfrag<DH>(ks, kb, f, lane, slot0);
                        s2[kk] = score(a, j, zero);
                    } else {
                        s2[kk] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
                    }
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
                for (int rt = 0; rt < RT; ++rt) o[j][rt] = mfma16x16x32(vtile(rt, sb), pb2, o[j][rt] * alpha);
            }
            lt = sum4(ll);
        }
        if (qb >= qend) continue;
        // v_rcp_f32 (1 ulp) rather than a correctly rounded division: the outputs are bf16
        const float inv = __builtin_amdgcn_rcpf(lt);
        uint16_t* dst = it.y0 + (uint32_t)(qb * sh.KSD * 512 + lane * 8);   // 32-bit offset in the item
        if constexpr (DH == 16) {
            u16x4 out;
#pragma unroll
            for (int i = 0; i < 4; ++i) out[i] = __builtin_bit_cast(uint16_t, (__bf16)(o[j][0][i] * inv));
            *reinterpret_cast<u16x4*>(dst + it.slot0) = out;
        } else {
#pragma unroll
            for (int f = 0; f < NF; ++f) {   // fragment f: O^T tiles 2f and 2f + 1
                const bf16x8 out = pack_b(o[j][2 * f] * inv, o[j][2 * f + 1] * inv);
                *reinterpret_cast<u16x8*>(dst + f * 512) = __builtin_bit_cast(u16x8, out);
            }
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
PWD_DEV void attn_passes(const AttnShape& sh, const AttnItem& it, int qbeg, int qend,
                         u16x8 (&qnext)[Frag<DH>::QMAX][Frag<DH>::NF], const bf16x8& ones, int lane) {
    constexpr int QM = Frag<DH>::QMAX, NF = Frag<DH>::NF;
    auto prefetch = [&](int qb_after) {
        if (qb_after < qend) load_q<NF, QM>(sh, it.q0, qb_after, qend, lane, qnext);
    };
    auto run = [&](auto qbc, int qb) {
        constexpr int QB = decltype(qbc)::value;
        u16x8 qv[QM][NF];
#pragma unroll
        for (int j = 0; j < QM; ++j)
#pragma unroll
            for (int f = 0; f < NF; ++f) qv[j][f] = qnext[j][f];
        prefetch(qb + QB);
        attn_pass<DH, QB>(sh, it, qb, qend, qv, ones, lane);
    };
    int qb = qbeg;
    for (; qend - qb >= QM; qb += QM) run(std::integral_constant<int, QM>{}, qb);
    if constexpr (QM > 2) {
        if (qend - qb >= 2) {
            run(std::integral_constant<int, 2>{}, qb);
            qb += 2;
        }
    }
    if (qend - qb == 1) run(std::integral_constant<int, 1>{}, qb);
}

// One workgroup per (window, head); K/V stay in LDS for the whole item. Workgroups of up to 4
// wavefronts share a CU (as many as their tiles fit in LDS); 8 wavefronts (tiles above 80 KB)
// keep two per SIMD on their own.
// Heads of 16 share their K/V fragments with the neighbouring head, so a workgroup stages
// the fragments once and runs both heads of the pair in turn.
template <int DH>
constexpr int heads_per_item() { return DH == 16 ? 2 : 1; }

template <int DH, int WAVES>
__global__ __launch_bounds__(WAVES * 64, WAVES == 8 ? 1 : 2) void attn_kernel(AttnParams p) {
    constexpr int NF = Frag<DH>::NF, QM = Frag<DH>::QMAX;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const AttnShape sh{p.N, p.nbw, p.H * DH / 32};
    const int nbw = sh.nbw;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t* ks = reinterpret_cast<uint16_t*>(smem);   // [nbw][NF][512]: K fragments
    uint16_t* vs = ks + (size_t)nbw * NF * 512;          // [nbw + 1][NF][512]: V tiles, + a zero block
    constexpr int HPI = heads_per_item<DH>();
    AttnItem it = make_item<DH>(p, sh, blockIdx.x * HPI);   // the pair's first head
    it.ks = ks;
    it.vs = vs;

    // Each wavefront owns a contiguous share of the query blocks; Q of its first pass is
    // loaded before the K/V staging, so its latency overlaps the staging.
    const int qbeg = wave * nbw / WAVES, qend = (wave + 1) * nbw / WAVES;
    u16x8 qnext[QM][NF];
    if (qbeg < qend) load_q<NF, QM>(sh, it.q0, qbeg, qend, lane, qnext);

    // stage K and V; an odd key-block count gets a zero V block so the last superblock's
    // missing keys meet P = 0 and V = 0
    stage_kv<NF>(sh, it.k0, ks, vs, wave, WAVES, lane);
    if (nbw & 1)
        for (int i = threadIdx.x; i < 256 * NF; i += blockDim.x)
            reinterpret_cast<uint32_t*>(vs + (size_t)nbw * NF * 512)[i] = 0u;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (qbeg < qend) {
        attn_passes<DH>(sh, it, qbeg, qend, qnext, ones_row(lane), lane);
        if constexpr (HPI == 2) {   // the pair's second head: its slots of the same fragments
            it.slot0 += 4;
            it.vhalf += 1;
            load_q<NF, QM>(sh, it.q0, qbeg, qend, lane, qnext);
            attn_passes<DH>(sh, it, qbeg, qend, qnext, ones_row(lane), lane);
        }
    }
}

template <int DH, int WAVES>
hipError_t launch_shape(const AttnParams& p, int nwin, hipStream_t s) {
    const size_t smem = attn_smem_bytes(DH, p.Npad, p.nbw);
    hipError_t e = hipFuncSetAttribute((const void*)attn_kernel<DH, WAVES>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    if (e != hipSuccess) return e;
    attn_kernel<DH, WAVES><<<dim3((unsigned)nwin * p.H / heads_per_item<DH>()), dim3(WAVES * 64), smem, s>>>(p);
    return hipGetLastError();
}

template <int DH>
hipError_t launch_dh(const AttnParams& p, int nwin, hipStream_t s) {
    // Wavefronts per (window, head). Heads of 16 and 32 (four query blocks per pass): as few
    // as keep two wavefronts per SIMD (8 per CU, the register limit) across the workgroups
    // whose tiles fit a CU's 160 KB of LDS, so that as many items as possible are in flight to
    // cover each other's K/V copies -- one where eight or more tiles fit (d11: 17 KB), two
    // where four do (d17: 37 KB, 9 % faster than four wavefronts; 168 tokens: 12 %), four for
    // two 79 KB tiles (d25). Heads of 64 (two query blocks per pass): enough wavefronts for a
    // pass each, at most four (two per item measured 8 % slower at 120 tokens). Either way a
    // tile above 80 KB leaves room for one workgroup, which gets eight wavefronts, and a
    // window of at most QMAX query blocks takes one.
    constexpr int QM = Frag<DH>::QMAX;
    const size_t tile = attn_smem_bytes(DH, p.Npad, p.nbw);
    const int fit = (int)(160 * 1024 / tile);
    if (p.nbw <= QM) return launch_shape<DH, 1>(p, nwin, s);
    if (QM >= 4 && fit >= 8) return launch_shape<DH, 1>(p, nwin, s);
    if (QM >= 4 ? fit >= 4 : p.nbw <= 2 * QM) return launch_shape<DH, 2>(p, nwin, s);
    if (ATTN_WIDE && tile > 80 * 1024) return launch_shape<DH, 8>(p, nwin, s);
    return launch_shape<DH, 4>(p, nwin, s);
}

}  // namespace

size_t attn_smem_bytes(int dh, int Npad, int nbw) {
    (void)Npad;
    // K [nbw] and V [nbw + 1] blocks of 1 KB fragments, two per block for a head of 64
    return (size_t)(2 * nbw + 1) * (dh == 64 ? 2 : 1) * 1024;
}

hipError_t launch_attn(int dh, const AttnParams& p, int nwin, hipStream_t s) {
    if (nwin <= 0) return hipSuccess;
    if (dh == 64) return launch_dh<64>(p, nwin, s);
    if (dh == 32) return launch_dh<32>(p, nwin, s);
    if (dh == 16) return launch_dh<16>(p, nwin, s);
    return hipErrorInvalidValue;
}
