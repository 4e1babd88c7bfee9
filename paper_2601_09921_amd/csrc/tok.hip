// Token-local stages of one Syndrome Transformer step, fused per token (bf16 MFMA path).
//
// One launch runs, for 32 tokens per wavefront, any of:
//   POST : out-projection of the attention output, residual, LayerNorm 1, feed-forward
//          D -> F -> D with ReLU, residual, LayerNorm 2 (App. A.2 Syndrome Transformer;
//          post-norm residual blocks).
//   EMBED: the stabilizer embedding of round t and the recurrent fold
//          X = kappa * (E_t w_e + b_e + PE + X) (App. A.1 embedder and positional
//          encoding; App. A.2 fold equation; Algorithm 1, D_0 = 0 at t = 0). With RESNET
//          the embedder's residual Conv1d block adds its output R, a function of the events
//          at the five cells around the token's cell (two kernel-3 layers) and of how close
//          the cell is to the ends of the flattened array, looked up in a host-built table.
//          Its input is one bit per cell lifted by Linear(1 -> D), so the lookup is exact.
//   QKV  : the Q, K, V projections of the following layer.
// With the dilated convolutions between LayerNorm 1 and the feed-forward, POST runs as two
// launches, WO (out-projection, residual, LayerNorm 1; it also writes the convolutions' input)
// and FFN (feed-forward, residual, LayerNorm 2, then EMBED / QKV as after POST), around the
// convolution units of conv_kernel at the end of this file.
// The residual stream stays fp32 in registers; only GEMM operands are rounded to bf16.
// GEMMs are transposed (Out^T = W^T In^T) so tokens lie along MFMA columns: LayerNorm
// reduces over the four lanes that share a token, and each accumulator becomes the next
// GEMM's B operand in registers.
//
// Weights reach the MFMAs through LDS: the host lays every weight fragment out in the exact
// order the kernel consumes them (a "weight stream"), and the workgroup pulls the stream
// through a double-buffered LDS ring in 32 KB chunks with direct global->LDS loads.
// The loads of chunk i+1 are interleaved with the fragment reads of chunk i, and the reads
// are software-pipelined in program order (a ring of fragments in flight ahead of the MFMAs).
// Every fragment read from LDS feeds 2 MFMAs of each wavefront (one per 16-token block the
// wavefront owns). Activations (X, Y, Q/K/V) are streamed with non-temporal accesses.
//
// With TOK_MX the Q/K/V projections and the feed-forward's first matrix run on MXFP8 operands
// with v_mfma_scale_f32_16x16x128_f8f6f4 (OCP Microscaling: E4M3 elements, one E8M0 scale per
// block of 32 reduction elements). That instruction pairs byte e of lane group g of A with
// byte e of lane group g of B, and lane group kb supplies the scale of K block kb, which is made
// of the first 16 bytes of lane groups 2 kb, 2 kb + 1 (kb < 2) or the last 16 bytes of lane
// groups 2 (kb - 2), 2 (kb - 2) + 1. A token's activations are quantized where they sit, in the
// C-fragment layout: lane (column n, group g) packs the 32 features 128 s + 16 r + 4 g + i
// (r = 0..7, i = 0..3) of 128-feature slice s as bytes 4 r + i, so the blocks of a slice are
// {16 r + 4 g + i : g in {2 p, 2 p + 1}, r in [4 h, 4 h + 4)} for block 2 h + p. A block's
// largest magnitude takes one lane-pair exchange; its owner lane gets it with one more. The
// weights are quantized by the host to the same blocks, one scale per output feature and
// block, and each 32 KB chunk carries its fragments' scales in one 1 KB slot.
#include "common.h"
#include "kernels.h"
#include "pipeline.h"

#include <type_traits>
#include <utility>

namespace {

constexpr int FRAG = 512;       // bf16 values per fragment (1 KB)

// Two 16-token blocks per wavefront and 4 wavefronts per workgroup, within 256 registers and
// 80 KB of LDS so that two workgroups share a CU: each SIMD runs two wavefronts, and one
// workgroup's activation loads, chunk barriers and stores overlap the other's MFMAs. (One
// 8-wavefront workgroup per CU, sharing one weight stream, measured 3-6 % slower.)
template <int D, int FLAGS>
constexpr int tok_waves() { return 4; }
constexpr int TB = 2;

template <int D, int NW, int MR>
struct Shape {
    static constexpr int CHUNK = 32;                  // weight fragments per LDS chunk
    static constexpr int RT = D / 16;                 // 16-row C tiles of a D-vector
    static constexpr int KS = D / 32;                 // 32-deep k-steps of a D-vector
    static constexpr int F = MR * D;                  // feed-forward width (MR = 4 or 5)
    static constexpr int CH = 8192 / D;               // hidden units per feed-forward chunk
    static constexpr int NMLP = F / CH;               // feed-forward sub-chunks (32 fragments each)
    static constexpr int MLP_PER = CHUNK / 32;        // feed-forward sub-chunks per LDS chunk
    static constexpr int MLP_CHUNKS = NMLP / MLP_PER;
    static constexpr int WO_CHUNKS = RT * KS / CHUNK;
    static constexpr int QKV_CHUNKS = (3 * D / 16) * KS / CHUNK;
    static constexpr int OG_PER_CHUNK = CHUNK / (2 * KS);
    static constexpr int POST_CHUNKS = WO_CHUNKS + MLP_CHUNKS;
    static_assert((CH / 16) * KS + RT * (CH / 32) == 32, "32 fragments per feed-forward sub-chunk");
    // MXFP8 (TOK_MX): 8-bit fragments of 16 rows x 128 k (2 KB, two 1 KB halves = two reads).
    // A feed-forward chunk holds the CH hidden units' W1 fragments (hidden row tile, k-step)
    // followed by their bf16 W2 fragments, a Q/K/V chunk 12 fragments (output group, k-step,
    // row tile); slot MX_SCALE_SLOT holds the chunk's weight scales, lane-major, byte j of a
    // lane for 8-bit fragment j; the other slots are unused.
    static constexpr int KS8 = D / 128;
    static constexpr int MX_SCALE_SLOT = 24;
    static constexpr int MX_NW1 = (CH / 16) * KS8;
    static constexpr int MX_FFN_READS = 2 * MX_NW1 + RT * (CH / 32);
    static constexpr int MX_QKV_FRAGS = 12;
    static constexpr int MX_OPC = MX_QKV_FRAGS / (2 * KS8);   // output groups per Q/K/V chunk
    static constexpr int MX_QKV_READS = 2 * MX_QKV_FRAGS;
    static constexpr int MX_QKV_CHUNKS = (3 * D / 32) / MX_OPC;
    static_assert(MX_FFN_READS == MX_SCALE_SLOT && MX_QKV_READS == MX_SCALE_SLOT, "data ahead of the scales");
    static_assert((3 * D / 32) % MX_OPC == 0 && MX_NW1 <= 4 && MLP_PER == 1, "MXFP8 chunk layout");
    static_assert(NMLP % MLP_PER == 0, "whole feed-forward chunks");
    static_assert(RT * KS % CHUNK == 0 && (3 * D / 16) * KS % CHUNK == 0, "whole chunks");
};

#ifndef TOK_NT
#define TOK_NT 1
#endif
// Activations are read and written once per launch; with TOK_NT their loads and stores are
// non-temporal so they do not push the weight stream out of the L2 cache.
template <typename T>
PWD_DEV T ld_stream(const T* p) {
    if constexpr (TOK_NT) return __builtin_nontemporal_load(p);
    else return *p;
}
template <typename T>
PWD_DEV void st_stream(T* p, T v) {
    if constexpr (TOK_NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}
// The token-major copy G of the dilated convolutions' input is stored through L2 (plain
// stores): one store instruction covers one k-step of 16 tokens, i.e. the 64-byte halves of 16
// 128-byte lines, whose other halves the next instruction writes. Through L2 the halves of a
// line combine before write-back; non-temporal stores sent them to memory separately (46 % more
// bytes written than G holds, and the out-projection launch that writes G 14 % slower).
template <typename T>
PWD_DEV void st_l2(T* p, T v) { *p = v; }

PWD_DEV bf16x8 ldfrag(const uint16_t* __restrict__ base, int64_t frag, int lane) {
    const u16x8 v = ld_stream(reinterpret_cast<const u16x8*>(base + (frag * 64 + lane) * 8));
    return __builtin_bit_cast(bf16x8, v);
}

PWD_DEV bf16x8 lds_frag(const uint16_t* buf, int j, int lane) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(buf + j * FRAG + lane * 8));
}

PWD_DEV void stfrag(uint16_t* __restrict__ base, int64_t frag, int lane, bf16x8 v) {
    st_stream(reinterpret_cast<u16x8*>(base + (frag * 64 + lane) * 8), __builtin_bit_cast(u16x8, v));
}


PWD_DEV u16x4 to_bf16x4(f32x4 v) {
    u16x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = __builtin_bit_cast(uint16_t, (__bf16)v[i]);
    return r;
}

PWD_DEV f32x4 relu4(f32x4 v) {
    f32x4 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = v[i] > 0.f ? v[i] : 0.f;
    return r;
}

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// ---- MXFP8 (TOK_MX)
// E8M0 scale of a block whose largest magnitude is m >= 0: 2^(floor(log2 m) - 8), 8 being the
// exponent of E4M3's largest power of two, as a biased byte (floor(log2 m) + 127 is m's own
// exponent field); 0 (2^-127) for m below 2^-119, zero included.
PWD_DEV uint32_t mx_scale_byte(float m) {
    const int e = (int)(__float_as_uint(m) >> 23) - 8;
    return e > 0 ? (uint32_t)e : 0u;
}
// 1 / scale, exactly: 2^(127 - byte) for byte in [0, 247]
PWD_DEV float mx_inv_scale(uint32_t byte) { return __uint_as_float((254u - byte) << 23); }
// Four values to E4M3 bytes (round to nearest, ties to even). The conversion does not
// saturate, so magnitudes are clamped to 448, E4M3's largest finite value, first.
PWD_DEV uint32_t e4m3x4(float a, float b, float c, float d) {
    const float lim = 448.f;
    const int w = __builtin_amdgcn_cvt_pk_fp8_f32(__builtin_amdgcn_fmed3f(a, -lim, lim),
                                                  __builtin_amdgcn_fmed3f(b, -lim, lim), 0, false);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(__builtin_amdgcn_fmed3f(c, -lim, lim),
                                                     __builtin_amdgcn_fmed3f(d, -lim, lim), w, true);
}

// MXFP8 B (or A) operands of each token from its fp32 C fragments: q[s][b] holds slice s of
// block b's token (bytes 4 r + i = feature 128 s + 16 r + 4 g + i), and byte b * KS8 + s of
// `scales` the E8M0 scale of K block g of that slice (the block this lane's scale stands for).
template <int RT, int TB>
PWD_DEV void quantize_mx(const f32x4 (&x)[RT][TB], i32x8 (&q)[RT / 8][TB], uint32_t& scales, int g) {
    constexpr int KS8 = RT / 8;
    static_assert(KS8 * TB <= 4, "scale bytes fit one register");
    scales = 0u;
#pragma unroll
    for (int b = 0; b < TB; ++b)
#pragma unroll
        for (int s = 0; s < KS8; ++s) {
            // largest magnitudes of this lane's two halves (r < 4, r >= 4), then of the lane pair
            // (groups 2 p, 2 p + 1) that forms each block
            float mlo = 0.f, mhi = 0.f;
#pragma unroll
            for (int r = 0; r < 8; ++r)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float a = fabsf(x[8 * s + r][b][i]);
                    if (r < 4) mlo = fmaxf(mlo, a);
                    else mhi = fmaxf(mhi, a);
                }
            float o;
            float t = swap16(mlo, o);
            mlo = fmaxf(t, o);
            t = swap16(mhi, o);
            mhi = fmaxf(t, o);
            // blocks of both pairs: *0 from groups {0, 1}, *1 from groups {2, 3}
            float lo1, hi1;
            const float lo0 = swap32(mlo, lo1);
            const float hi0 = swap32(mhi, hi1);
            const float owned = g == 0 ? lo0 : g == 1 ? lo1 : g == 2 ? hi0 : hi1;
            scales |= mx_scale_byte(owned) << (8 * (b * KS8 + s));
            const float ilo = mx_inv_scale(mx_scale_byte(mlo)), ihi = mx_inv_scale(mx_scale_byte(mhi));
#pragma unroll
            for (int r = 0; r < 8; ++r) {
                const float inv = r < 4 ? ilo : ihi;
                const f32x4 v = x[8 * s + r][b];
                q[s][b][r] = (int)e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
            }
        }
}

// An 8-bit fragment from its two 1 KB halves (bytes 0-15 and 16-31 of each lane).
PWD_DEV i32x8 join_halves(const bf16x8& lo, const bf16x8& hi) {
    const i32x4 a = __builtin_bit_cast(i32x4, lo), b = __builtin_bit_cast(i32x4, hi);
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// D = scale_a scale_b (A B) + C on MXFP8 operands; byte ia of sa and byte ib of sb are the
// E8M0 scales of this lane's A row / B column block. ia and ib fold to constants in the
// unrolled callers (the instruction takes the byte selectors as immediates).
template <int IA, int IB>
PWD_DEV f32x4 mfma_mx_sel(const i32x8& a, const i32x8& b, f32x4 c, uint32_t sa, uint32_t sb) {
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, IA, (int)sa, IB, (int)sb);
}
PWD_DEV f32x4 mfma_mx(const i32x8& a, const i32x8& b, f32x4 c, uint32_t sa, int ia, uint32_t sb, int ib) {
    switch (ia * 4 + ib) {
#define PWD_MX_CASE(k) case k: return mfma_mx_sel<k / 4, k % 4>(a, b, c, sa, sb);
        PWD_MX_CASE(0) PWD_MX_CASE(1) PWD_MX_CASE(2) PWD_MX_CASE(3) PWD_MX_CASE(4) PWD_MX_CASE(5)
        PWD_MX_CASE(6) PWD_MX_CASE(7) PWD_MX_CASE(8) PWD_MX_CASE(9) PWD_MX_CASE(10) PWD_MX_CASE(11)
        PWD_MX_CASE(12) PWD_MX_CASE(13) PWD_MX_CASE(14)
#undef PWD_MX_CASE
        default: return mfma_mx_sel<3, 3>(a, b, c, sa, sb);
    }
}

// Look-ahead of the fragment reads (fragments in flight ahead of the MFMAs that use them);
// with two wavefronts per SIMD a short ring suffices and keeps within 256 registers.
#ifndef TOK_LA_WO
#define TOK_LA_WO 4
#endif
#ifndef TOK_LA_MLP
#define TOK_LA_MLP 4
#endif
#ifndef TOK_LA_QKV
#define TOK_LA_QKV 4
#endif
// Spacing, in fragment reads, of the next chunk's loads (0: spread over the whole chunk).
#ifndef TOK_DMA_SP
#define TOK_DMA_SP 2
#endif

// The two LDS buffers of the weight stream. They are separate objects so the compiler can
// tell that the direct-to-LDS prefetch into one never aliases reads of the other.
template <int PAR, int CHUNK>
PWD_DEV uint16_t* wbuf() {
    __shared__ __align__(16) uint16_t buf[CHUNK * FRAG];   // one object per (buffer, size)
    return buf;
}

// The weight stream of one launch: `post` chunks first, then `qkv` chunks, pulled through
// the two LDS buffers (chunk i lives in buffer i % 2). sync<i % 2>(i) makes chunk i visible
// to every wavefront. While the wavefronts compute on chunk i, the CHUNK / NW fragments
// of chunk i+1 that each wavefront loads go out one at a time between its fragment reads
// (after_read), rather than in one burst, so LDS reads and direct-to-LDS writes do not queue
// behind each other. The last chunk reloads itself into the idle buffer so that the loads
// stay branch-free; the kernel waits for them before it ends.
template <int CHUNK, int NW>
struct WeightPipe {
    static constexpr int PER_WAVE = CHUNK / NW;
    const uint16_t* post;
    const uint16_t* qkv;
    int n_post, total;
    int wave;            // wavefront index, wavefront-uniform
    int lane;

    __device__ const uint16_t* src(int i) const {
        return i < n_post ? post + (size_t)i * CHUNK * FRAG : qkv + (size_t)(i - n_post) * CHUNK * FRAG;
    }
    // source of the chunk loaded while chunk i is in use
    __device__ const uint16_t* next(int i) const { return src(i + 1 < total ? i + 1 : i); }

    // Fragment f of the chunk at `s` into fragment slot f of buffer PAR (one 1 KB direct
    // load; awaited in sync() and at kernel end).
    template <int PAR>
    __device__ void part(const uint16_t* s, int j) const {
        const int f = wave * PER_WAVE + j;
        lds_load_1k(uniform_ptr(s + f * FRAG), lds_addr(wbuf<PAR, CHUNK>() + f * FRAG), lane);
    }
    template <int PAR>
    __device__ void issue(int i) const {
#pragma unroll
        for (int j = 0; j < PER_WAVE; ++j) part<PAR>(src(i), j);
    }
    // Runs after fragment read r of a chunk of NREAD reads pipelined with look-ahead LA: the
    // PER_WAVE loads of the next chunk follow reads LA, LA + SP, LA + 2 SP, ...
    template <int NREAD, int LA>
    static constexpr int spacing() {
        constexpr int SP_MAX = PER_WAVE > 1 ? (NREAD - 1 - LA) / (PER_WAVE - 1) : 1;
        return TOK_DMA_SP > 0 && TOK_DMA_SP < SP_MAX ? TOK_DMA_SP : SP_MAX;
    }
    // Read index after which the last load of the next chunk is issued.
    template <int NREAD, int LA>
    static constexpr int last_load_read() { return LA + spacing<NREAD, LA>() * (PER_WAVE - 1); }

    template <int PAR, int NREAD, int LA>
    __device__ void after_read(const uint16_t* s, int r) const {
        constexpr int SP = spacing<NREAD, LA>();
        static_assert(SP >= 1, "loads fit in the chunk");
        if (r >= LA && (r - LA) % SP == 0 && (r - LA) / SP < PER_WAVE) part<PAR>(s, (r - LA) / SP);
    }
    // Chunk i becomes visible to every wavefront. Vector memory operations retire in issue
    // order, so this wavefront's loads of chunk i have landed once at most YOUNGER of its
    // vector memory operations are outstanding: YOUNGER counts what it issued after its last
    // load of chunk i (global stores), which therefore need not complete here.
    template <int PAR, int YOUNGER>
    __device__ const uint16_t* sync(int) const {
        static_assert(YOUNGER >= 0 && YOUNGER < 64, "vmcnt range");
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"(YOUNGER) : "memory");
        __syncthreads();                                   // everyone's part landed; buffer i-1 is free
        return wbuf<PAR, CHUNK>();
    }
};

// LDS of one workgroup (two per CU): the weight ring (two 32-fragment buffers) + vectors.
constexpr int LDS_BUDGET = 80 * 1024, RING_BYTES = 2 * 32 * FRAG * 2;

// b_v is stored with each value four times (the bias of a V tile is one column value per
// lane, loaded as the f32x4 an accumulator starts from) where that fits in LDS, else once.
constexpr int bv_rep(int D, int F) { return (12 * D + F) * 4 + RING_BYTES <= LDS_BUDGET ? 4 : 1; }

// Per-launch vectors staged in LDS once: [bo g1 be1 b2 g2 be2 | b1 (F) | b_q b_k | b_v].
template <int D, int F>
struct Vecs {
    static constexpr int BO = 0, G1 = D, BE1 = 2 * D, B2 = 3 * D, G2 = 4 * D, BE2 = 5 * D;
    static constexpr int REP = bv_rep(D, F);
    static constexpr int B1 = 6 * D, BQKV = 6 * D + F, BV = BQKV + 2 * D, QKV_VECS = (2 + REP) * D;
    static constexpr int SIZE = BQKV + QKV_VECS;
    static_assert(SIZE * 4 + RING_BYTES <= LDS_BUDGET, "vector table fits");
};

// Global stores a wavefront issues in one Q/K/V chunk after its last load of the next
// chunk. Output group o2 is stored in the MFMA step of its last fragment read,
// r = (o2 + 1) * 2 KS - 1, which follows the loads issued after reads up to r + LA - 1.
template <int CHUNK, int NW, int KS, int LA, int STORES_PER_GROUP>
constexpr int qkv_stores_after_last_load() {
    constexpr int LAST = WeightPipe<CHUNK, NW>::template last_load_read<CHUNK, LA>();
    int n = 0;
    for (int o2 = 0; o2 < CHUNK / (2 * KS); ++o2)
        if ((o2 + 1) * 2 * KS - 1 + LA - 1 >= LAST) n += STORES_PER_GROUP;
    return n;
}

// The same for a Q/K/V chunk of the MXFP8 layout: its output group o2 is stored after read
// (o2 + 1) * 4 KS8 - 1; groups of Q and K store TB fragments, groups of V 2 TB half-fragments
// (one chunk may hold both kinds).
template <int D, int NW, int LA>
constexpr int mx_qkv_stores_after_last_load(int qc) {
    using S = Shape<D, NW, 4>;
    constexpr int LAST = WeightPipe<S::CHUNK, NW>::template last_load_read<S::MX_QKV_READS, LA>();
    int n = 0;
    for (int o2 = 0; o2 < S::MX_OPC; ++o2)
        if ((o2 + 1) * 4 * S::KS8 - 1 + LA - 1 >= LAST) n += qc * S::MX_OPC + o2 >= 2 * S::KS ? 2 * TB : TB;
    return n;
}

template <int D, int MR, int FLAGS>
__global__ __launch_bounds__((tok_waves<D, FLAGS>() * 64), 2) void tok_kernel(TokParams p) {
    constexpr int WAVES = tok_waves<D, FLAGS>();
    using S = Shape<D, WAVES, MR>;
    constexpr int LA_WO = TOK_LA_WO, LA_MLP = TOK_LA_MLP, LA_QKV = TOK_LA_QKV;
    using V = Vecs<D, S::F>;
    constexpr int RT = S::RT, KS = S::KS, CH = S::CH;
    // DO_WO: out-projection + LN1; DO_FFN: feed-forward + LN2; POST: either (X is loaded)
    constexpr bool WO_ONLY = (FLAGS & TOK_WO) != 0, FFN_ONLY = (FLAGS & TOK_FFN) != 0;
    static_assert(!WO_ONLY || FLAGS == TOK_WO, "the out-projection-only launch stands alone");
    constexpr bool DO_WO = (FLAGS & TOK_POST) != 0 || WO_ONLY, DO_FFN = (FLAGS & TOK_POST) != 0 || FFN_ONLY;
    constexpr bool POST = DO_WO || DO_FFN, QKV = (FLAGS & TOK_QKV) != 0;
    constexpr bool MX = (FLAGS & TOK_MX) != 0;
    static_assert(!MX || (!WO_ONLY && !FFN_ONLY), "MXFP8 runs without the dilated convolutions");
    constexpr int KS8 = S::KS8;
    constexpr int WO_CH = DO_WO ? S::WO_CHUNKS : 0, N_POST = WO_CH + (DO_FFN ? S::MLP_CHUNKS : 0);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int g = lane >> 4;
    const int col = lane & 15;
    const int64_t tb0 = ((int64_t)blockIdx.x * WAVES + wave) * TB;

    constexpr int CHUNK = S::CHUNK;
    WeightPipe<CHUNK, WAVES> pipe;
    pipe.post = DO_WO ? p.post_stream : p.post_stream + (size_t)S::WO_CHUNKS * CHUNK * FRAG;
    pipe.qkv = p.qkv_stream;
    pipe.n_post = N_POST;
    pipe.total = pipe.n_post + (QKV ? (MX ? S::MX_QKV_CHUNKS : S::QKV_CHUNKS) : 0);
    pipe.wave = __builtin_amdgcn_readfirstlane(wave);
    pipe.lane = lane;

    // The activations come from HBM and are issued first, so their latency overlaps that of
    // the first weight chunk and of the vector staging below (all of it is awaited at the
    // first chunk's sync).
    f32x4 x[RT][TB];
    bf16x8 y[DO_WO ? KS : 1][TB];
    if constexpr (POST) {
        if constexpr (DO_WO) {
#pragma unroll
            for (int b = 0; b < TB; ++b)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) y[ks][b] = ldfrag(p.Y, (tb0 + b) * KS + ks, lane);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int b = 0; b < TB; ++b)
                x[rt][b] = ld_stream(reinterpret_cast<const f32x4*>(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4));
    }
    pipe.template issue<0>(0);

    // detection events of round t for this lane's token of each block (EMBED), computed while
    // few registers are live
    constexpr bool RES = (FLAGS & TOK_RESNET) != 0;
    static_assert(!RES || (FLAGS & TOK_EMBED) != 0, "the residual block is part of the embedding");
    float ev[TB];
    int row[TB];   // RESNET: the token's row of the block's table
    if constexpr ((FLAGS & TOK_EMBED) != 0) {
#pragma unroll
        for (int b = 0; b < TB; ++b) {
            const int64_t tb = tb0 + b;
            const int64_t w = tb / p.nbw;
            const int s = (int)(tb - w * p.nbw) * 16 + col;   // token
            ev[b] = 0.f;
            row[b] = 0;
            const int st = s < p.ntok ? (p.tok_stab ? p.tok_stab[s] : s) : -1;   // its stabilizer
            if (w < p.in.nwin) {
                const uint32_t* m = p.in.meas + w * (int64_t)(p.in.W + 1) * p.in.words;
                const int type = p.in.types[w];
                auto bit = [&](int q) -> uint32_t {   // event of stabilizer q in round t
                    const uint32_t word = event_word(m, p.in.words, p.t, q >> 5, type, p.in.b_left, p.in.d);
                    return (word >> (q & 31)) & 1u;
                };
                if (st >= 0) ev[b] = (float)bit(st);
                if constexpr (RES) {
                    if (s < p.ntok) {
                        const int* nb = p.emb_nb + (size_t)s * 8;
                        uint32_t pat = 0u;
#pragma unroll
                        for (int j = 0; j < 5; ++j) {
                            const int q = nb[j];
                            if (q >= 0) pat |= bit(q) << j;
                        }
                        row[b] = nb[5] * 32 + (int)pat;
                    }
                }
            }
        }
    }

    // Per-launch vectors, staged in LDS by direct loads of 256 bytes (64 lanes x 4 bytes):
    // vec[0, 6 D + F) from the POST layer's vector table, then the Q/K/V biases. The first
    // chunk's sync awaits and publishes them.
    __shared__ __align__(16) float vec[V::SIZE];
    {
        constexpr int NP_V = POST ? V::BQKV / 64 : 0, NQ_V = QKV ? V::QKV_VECS / 64 : 0;
        static_assert(V::BQKV % 64 == 0 && V::QKV_VECS % 64 == 0, "whole 256-byte pieces");
        for (int k = pipe.wave; k < NP_V + NQ_V; k += WAVES) {
            const float* src = k < NP_V ? p.post_vecs + k * 64 : p.bqkv + (k - NP_V) * 64;
            const int dst = k < NP_V ? k * 64 : V::BQKV + (k - NP_V) * 64;
            // (inline assembly for the reason given at lds_load_1k)
            asm volatile(LDS_DMA_GUARD "global_load_lds_dword %0, %1" :: "v"((uint32_t)lane * 4), "s"(uniform_ptr(src)),
                         "{m0}"(lds_addr(vec + dst)) : "memory");
        }
    }

    if constexpr (DO_WO) {
        // ---- out-projection + residual + LayerNorm 1; accumulators start at X (+ b_o below)
        {
            constexpr int LA = LA_WO;
            auto wo_chunk = [&](auto par, int c) {
                constexpr int PAR = decltype(par)::value;
                const uint16_t* buf = pipe.template sync<PAR, 0>(c);
                const uint16_t* nx = pipe.next(c);
                pipelined<CHUNK, LA>(
                    [&](int r) { return lds_frag(buf, r, lane); },
                    [&](int r, const bf16x8& a) {
                        const int fr = c * CHUNK + r, rt = fr / KS, ks = fr % KS;
#pragma unroll
                        for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, y[ks][b], x[rt][b]);
                    },
                    [&](int r) { pipe.template after_read<1 - PAR, CHUNK, LA>(nx, r); });
                sched_pipeline<CHUNK, TB, LA>();
            };
            static_assert(S::WO_CHUNKS == 1 || S::WO_CHUNKS % 2 == 0, "Wo chunks");
            if constexpr (S::WO_CHUNKS == 1) {
                wo_chunk(std::integral_constant<int, 0>{}, 0);
            } else {
#pragma unroll
                for (int c = 0; c < S::WO_CHUNKS; c += 2) {
                    wo_chunk(std::integral_constant<int, 0>{}, c);
                    wo_chunk(std::integral_constant<int, 1>{}, c + 1);
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
    }
    if constexpr (WO_ONLY) {
        // the dilated convolutions' input: each token's B fragments, token-major
#pragma unroll
        for (int b = 0; b < TB; ++b)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                st_l2(reinterpret_cast<u16x8*>(p.G + ((((tb0 + b) * 16 + col) * KS + ks) * 4 + g) * 8),
                          __builtin_bit_cast(u16x8, pack_b(x[2 * ks][b], x[2 * ks + 1][b])));
    }
    if constexpr (DO_FFN) {
        if constexpr (!DO_WO) {
            // no chunk sync has run yet: await and publish the staged vectors (b_2 below)
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
        }
        // ---- feed-forward, hidden units in chunks of CH; accumulators start at X + b_2
        bf16x8 xb[MX ? 1 : KS][TB];
        i32x8 xq[MX ? KS8 : 1][TB];   // MX: the LayerNorm output in MXFP8 ...
        uint32_t sx = 0u;             // ... and its scales
        if constexpr (MX) {
            quantize_mx<RT, TB>(x, xq, sx, g);
        } else {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
#pragma unroll
                for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 bias = ld4(vec + V::B2 + rt * 16 + 4 * g);
#pragma unroll
            for (int b = 0; b < TB; ++b) x[rt][b] += bias;
        }
        // One LDS chunk holds MP feed-forward sub-chunks of CH hidden units, each 32 fragments:
        // (CH / 16) * KS fragments of W1 (hidden = W1^T x), then RT * (CH / 32) of W2
        // (x += W2^T relu(hidden)).
        constexpr int MP = S::MLP_PER;
        constexpr int LA = LA_MLP;
        constexpr int NW1 = (CH / 16) * KS;
        auto mlp_chunk = [&](auto par, int c) {
            constexpr int PAR = decltype(par)::value;
            const int ci = WO_CH + c;
            const uint16_t* buf = pipe.template sync<PAR, 0>(ci);
            f32x4 h[MP][CH / 16][TB];
#pragma unroll
            for (int u = 0; u < MP; ++u)
#pragma unroll
                for (int rh = 0; rh < CH / 16; ++rh) {
                    const f32x4 bias = ld4(vec + V::B1 + (c * MP + u) * CH + rh * 16 + 4 * g);
#pragma unroll
                    for (int b = 0; b < TB; ++b) h[u][rh][b] = bias;
                }
            const uint16_t* nx = pipe.next(ci);
            __builtin_amdgcn_sched_barrier(0);
            bf16x8 hb[MP][CH / 32][TB];
            pipelined<MP * 32, LA>(
                [&](int r) { return lds_frag(buf, r, lane); },
                [&](int r, const bf16x8& a) {
                    const int u = r / 32, k = r % 32;
                    if (k < NW1) {
                        const int rh = k / KS, ks = k % KS;
#pragma unroll
                        for (int b = 0; b < TB; ++b) h[u][rh][b] = mfma16x16x32(a, xb[ks][b], h[u][rh][b]);
                        if (k == NW1 - 1) {
#pragma unroll
                            for (int kh = 0; kh < CH / 32; ++kh)
#pragma unroll
                                for (int b = 0; b < TB; ++b)
                                    hb[u][kh][b] = pack_b(relu4(h[u][2 * kh][b]), relu4(h[u][2 * kh + 1][b]));
                        }
                    } else {
                        const int rt = (k - NW1) / (CH / 32), kh = (k - NW1) % (CH / 32);
#pragma unroll
                        for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, hb[u][kh][b], x[rt][b]);
                    }
                },
                [&](int r) { pipe.template after_read<1 - PAR, MP * 32, LA>(nx, r); });
            sched_pipeline<MP * 32, TB, LA>();
        };
        // MX: the chunk's MX_NW1 8-bit W1 fragments (hidden row tile, k-step; two reads each)
        // against the quantized LayerNorm output, then its bf16 W2 fragments as above
        auto mlp_chunk_mx = [&](auto par, int c) {
            constexpr int PAR = decltype(par)::value;
            constexpr int NR = S::MX_FFN_READS, NP1 = 2 * S::MX_NW1;
            const int ci = WO_CH + c;
            const uint16_t* buf = pipe.template sync<PAR, 0>(ci);
            f32x4 h[CH / 16][TB];
#pragma unroll
            for (int rh = 0; rh < CH / 16; ++rh) {
                const f32x4 bias = ld4(vec + V::B1 + c * CH + rh * 16 + 4 * g);
#pragma unroll
                for (int b = 0; b < TB; ++b) h[rh][b] = bias;
            }
            const uint32_t wsc = *reinterpret_cast<const uint32_t*>(buf + S::MX_SCALE_SLOT * FRAG + lane * 8);
            const uint16_t* nx = pipe.next(ci);
            __builtin_amdgcn_sched_barrier(0);
            bf16x8 hb[CH / 32][TB];
            bf16x8 half0;
            pipelined<NR, LA>(
                [&](int r) { return lds_frag(buf, r, lane); },
                [&](int r, const bf16x8& a) {
                    if (r < NP1) {
                        if ((r & 1) == 0) {
                            half0 = a;
                            return;
                        }
                        const int j = r >> 1, rh = j / KS8, ks8 = j % KS8;
                        const i32x8 w = join_halves(half0, a);
#pragma unroll
                        for (int b = 0; b < TB; ++b) h[rh][b] = mfma_mx(w, xq[ks8][b], h[rh][b], wsc, j, sx, b * KS8 + ks8);
                        if (j == S::MX_NW1 - 1) {
#pragma unroll
                            for (int kh = 0; kh < CH / 32; ++kh)
#pragma unroll
                                for (int b = 0; b < TB; ++b)
                                    hb[kh][b] = pack_b(relu4(h[2 * kh][b]), relu4(h[2 * kh + 1][b]));
                        }
                    } else {
                        const int k = r - NP1, rt = k / (CH / 32), kh = k % (CH / 32);
#pragma unroll
                        for (int b = 0; b < TB; ++b) x[rt][b] = mfma16x16x32(a, hb[kh][b], x[rt][b]);
                    }
                },
                [&](int r) { pipe.template after_read<1 - PAR, NR, LA>(nx, r); });
            sched_pipeline_pairs<NR, TB, LA, NP1>();
        };
        static_assert(S::MLP_CHUNKS % 2 == 0, "feed-forward chunks come in pairs");
        constexpr int P0 = WO_CH & 1;
        for (int c = 0; c < S::MLP_CHUNKS; c += 2) {
            if constexpr (MX) {
                mlp_chunk_mx(std::integral_constant<int, P0>{}, c);
                mlp_chunk_mx(std::integral_constant<int, 1 - P0>{}, c + 1);
            } else {
                mlp_chunk(std::integral_constant<int, P0>{}, c);
                mlp_chunk(std::integral_constant<int, 1 - P0>{}, c + 1);
            }
        }
        layer_norm<RT, TB>(x, vec + V::G2, vec + V::BE2, p.eps, g);
    }

    if constexpr (DO_FFN && (FLAGS & TOK_EMBED) != 0) {
        // the state D_t itself, for a readout of this round (bf16, the readout's operand type)
        if (p.state_out) {
#pragma unroll
            for (int b = 0; b < TB; ++b)
#pragma unroll
                for (int rt = 0; rt < RT; ++rt)
                    st_stream(reinterpret_cast<u16x4*>(p.state_out + (((tb0 + b) * RT + rt) * 64 + lane) * 4),
                              to_bf16x4(x[rt][b]));
        }
    }
    if constexpr ((FLAGS & TOK_EMBED) != 0) {
        // ---- embedding of round t folded into the state: X = kappa (S_t + X)
#pragma unroll
        for (int b = 0; b < TB; ++b) {
            const int64_t tb = tb0 + b;
            const int blk = (int)(tb % p.nbw);
            const bool real = blk * 16 + col < p.ntok;
            const float e = ev[b];
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                f32x4 s0 = ld4(p.S0 + (((int64_t)blk * RT + rt) * 64 + lane) * 4);
                const f32x4 we = ld4(p.we + rt * 16 + 4 * g);
                if constexpr (RES) s0 += ld4(p.emb_tab + (size_t)row[b] * D + rt * 16 + 4 * g);
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
                st_stream(reinterpret_cast<f32x4*>(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4), x[rt][b]);
    };

    store_x();
    if constexpr (QKV && !MX) {
        bf16x8 xb[KS][TB];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int b = 0; b < TB; ++b) xb[ks][b] = pack_b(x[2 * ks][b], x[2 * ks + 1][b]);
        // 3D output features in groups of 32 (= one B fragment of Q, K or V)
        constexpr int NP = N_POST;
        constexpr int OPC = S::OG_PER_CHUNK;
        constexpr int LA = LA_QKV;
        // Q and K are stored as B fragments of their transposes (one 1 KB store per group and
        // token block); V as two 16x16 tiles with tokens as rows (its MFMA takes the
        // activations as the A operand), each 512 B, which the attention kernel copies to LDS
        // unchanged as the A fragments of V^T.
        constexpr int NQK = 2 * S::QKV_CHUNKS / 3;
        static_assert(S::QKV_CHUNKS % 3 == 0, "Q, K and V in whole chunks");
        constexpr int STORES_QK = qkv_stores_after_last_load<CHUNK, WAVES, KS, LA, TB>();
        constexpr int STORES_V = qkv_stores_after_last_load<CHUNK, WAVES, KS, LA, 2 * TB>();
        auto qkv_chunk = [&](auto qcc) {
            constexpr int qc = decltype(qcc)::value;
            constexpr int PAR = (NP + qc) & 1;
            constexpr bool VOUT = qc >= NQK;
            // before the first QKV chunk, the residual stream store (RT * TB stores) follows
            // the last load of this chunk; later, the previous chunk's output stores do
            constexpr int YOUNGER = qc == 0 ? RT * TB : (qc - 1 >= NQK ? STORES_V : STORES_QK);
            const uint16_t* buf = pipe.template sync<PAR, YOUNGER>(NP + qc);
            // fragment r = (o2 * KS + ks) * 2 + hh: rows 16 hh .. 16 hh + 15 of output group
            // qc * OPC + o2, k-step ks
            f32x4 q[OPC][2][TB];
#pragma unroll
            for (int o2 = 0; o2 < OPC; ++o2)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    if constexpr (VOUT) {   // bias along the tile's columns: lane col's value x 4
                        const int o = (qc * OPC + o2 - 2 * KS) * 32 + hh * 16 + col;
                        f32x4 bias;
                        if constexpr (V::REP == 4) {
                            bias = ld4(vec + V::BV + o * 4);
                        } else {
                            const float bv = vec[V::BV + o];
                            bias = f32x4{bv, bv, bv, bv};
                        }
#pragma unroll
                        for (int b = 0; b < TB; ++b) q[o2][hh][b] = bias;
                    } else {
                        const f32x4 bias = ld4(vec + V::BQKV + (qc * OPC + o2) * 32 + hh * 16 + 4 * g);
#pragma unroll
                        for (int b = 0; b < TB; ++b) q[o2][hh][b] = bias;
                    }
                }
            const uint16_t* nx = pipe.next(NP + qc);
            __builtin_amdgcn_sched_barrier(0);
            pipelined<CHUNK, LA>(
                [&](int r) { return lds_frag(buf, r, lane); },
                [&](int r, const bf16x8& a) {
                    const int hh = r & 1, ks = (r >> 1) % KS, o2 = (r >> 1) / KS;
#pragma unroll
                    for (int b = 0; b < TB; ++b) {
                        if constexpr (VOUT) q[o2][hh][b] = mfma16x16x32(xb[ks][b], a, q[o2][hh][b]);
                        else q[o2][hh][b] = mfma16x16x32(a, xb[ks][b], q[o2][hh][b]);
                    }
                    if (hh == 1 && ks == KS - 1) {
                        const int og = qc * OPC + o2;
#pragma unroll
                        for (int b = 0; b < TB; ++b) {
                            if constexpr (VOUT) {
                                uint16_t* t = p.QKV + ((tb0 + b) * (3 * KS) + og) * FRAG + lane * 4;
#pragma unroll
                                for (int h2 = 0; h2 < 2; ++h2)
                                    st_stream(reinterpret_cast<u16x4*>(t + h2 * (FRAG / 2)), to_bf16x4(q[o2][h2][b]));
                            } else {
                                const float sc = og < KS ? p.qscale : 1.0f;   // Q: log2(e)/sqrt(dh)
                                stfrag(p.QKV, (tb0 + b) * (3 * KS) + og, lane,
                                       pack_b(q[o2][0][b] * sc, q[o2][1][b] * sc));
                            }
                        }
                    }
                },
                [&](int r) { pipe.template after_read<1 - PAR, CHUNK, LA>(nx, r); });
            sched_pipeline<CHUNK, TB, LA>();
        };
        static_for<S::QKV_CHUNKS>(qkv_chunk);
    }
    if constexpr (QKV && MX) {
        // MXFP8: the residual stream quantized per token, then per chunk MX_OPC output groups of
        // 32 features, each KS8 k-steps x 2 row tiles of 8-bit fragments (two reads each);
        // Q and K as in the bf16 path, V with the activations as the A operand. A chunk may
        // hold groups of both kinds.
        i32x8 xq[KS8][TB];
        uint32_t sx;
        quantize_mx<RT, TB>(x, xq, sx, g);
        constexpr int NP = N_POST;
        constexpr int OPC = S::MX_OPC;
        constexpr int LA = LA_QKV;
        constexpr int NR = S::MX_QKV_READS;
        auto qkv_chunk = [&](auto qcc) {
            constexpr int qc = decltype(qcc)::value;
            constexpr int PAR = (NP + qc) & 1;
            constexpr int YOUNGER = qc == 0 ? RT * TB : mx_qkv_stores_after_last_load<D, WAVES, LA>(qc - 1);
            const uint16_t* buf = pipe.template sync<PAR, YOUNGER>(NP + qc);
            f32x4 q[OPC][2][TB];
#pragma unroll
            for (int o2 = 0; o2 < OPC; ++o2)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh) {
                    const int og = qc * OPC + o2;
                    f32x4 bias;
                    if (og >= 2 * KS) {   // V: bias along the tile's columns
                        const int o = (og - 2 * KS) * 32 + hh * 16 + col;
                        if constexpr (V::REP == 4) {
                            bias = ld4(vec + V::BV + o * 4);
                        } else {
                            const float bv = vec[V::BV + o];
                            bias = f32x4{bv, bv, bv, bv};
                        }
                    } else {
                        bias = ld4(vec + V::BQKV + og * 32 + hh * 16 + 4 * g);
                    }
#pragma unroll
                    for (int b = 0; b < TB; ++b) q[o2][hh][b] = bias;
                }
            const u32x4 wsc = *reinterpret_cast<const u32x4*>(buf + S::MX_SCALE_SLOT * FRAG + lane * 8);
            const uint16_t* nx = pipe.next(NP + qc);
            __builtin_amdgcn_sched_barrier(0);
            bf16x8 half0;
            pipelined<NR, LA>(
                [&](int r) { return lds_frag(buf, r, lane); },
                [&](int r, const bf16x8& a) {
                    if ((r & 1) == 0) {
                        half0 = a;
                        return;
                    }
                    // 8-bit fragment j = (o2 * KS8 + ks8) * 2 + hh
                    const int j = r >> 1, hh = j & 1, ks8 = (j >> 1) % KS8, o2 = (j >> 1) / KS8;
                    const int og = qc * OPC + o2;
                    const bool vout = og >= 2 * KS;
                    const i32x8 w = join_halves(half0, a);
#pragma unroll
                    for (int b = 0; b < TB; ++b) {
                        if (vout) q[o2][hh][b] = mfma_mx(xq[ks8][b], w, q[o2][hh][b], sx, b * KS8 + ks8, wsc[j >> 2], j & 3);
                        else q[o2][hh][b] = mfma_mx(w, xq[ks8][b], q[o2][hh][b], wsc[j >> 2], j & 3, sx, b * KS8 + ks8);
                    }
                    if (hh == 1 && ks8 == KS8 - 1) {
#pragma unroll
                        for (int b = 0; b < TB; ++b) {
                            if (vout) {
                                uint16_t* t = p.QKV + ((tb0 + b) * (3 * KS) + og) * FRAG + lane * 4;
#pragma unroll
                                for (int h2 = 0; h2 < 2; ++h2)
                                    st_stream(reinterpret_cast<u16x4*>(t + h2 * (FRAG / 2)), to_bf16x4(q[o2][h2][b]));
                            } else {
                                const float sc = og < KS ? p.qscale : 1.0f;   // Q: log2(e)/sqrt(dh)
                                stfrag(p.QKV, (tb0 + b) * (3 * KS) + og, lane,
                                       pack_b(q[o2][0][b] * sc, q[o2][1][b] * sc));
                            }
                        }
                    }
                },
                [&](int r) { pipe.template after_read<1 - PAR, NR, LA>(nx, r); });
            sched_pipeline_pairs<NR, TB, LA, NR>();
        };
        static_for<S::MX_QKV_CHUNKS>(qkv_chunk);
    }
    // The last chunk's reload into the idle buffer must land before the workgroup's LDS is
    // freed; the global stores issued after it need not.
    constexpr int END_YOUNGER = !QKV ? RT * TB + (WO_ONLY ? KS * TB : 0)
                              : MX   ? mx_qkv_stores_after_last_load<D, WAVES, LA_QKV>(S::MX_QKV_CHUNKS - 1)
                                     : qkv_stores_after_last_load<CHUNK, WAVES, KS, LA_QKV, 2 * TB>();
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(END_YOUNGER) : "memory");
}

template <int D, int MR, int FLAGS>
void launch_variant(const TokParams& p, int64_t n_tb, hipStream_t s) {
    constexpr int WAVES = tok_waves<D, FLAGS>();
    const int64_t per_wg = (int64_t)WAVES * TB;
    const dim3 grid((unsigned)((n_tb + per_wg - 1) / per_wg)), block(WAVES * 64);
    tok_kernel<D, MR, FLAGS><<<grid, block, 0, s>>>(p);
}

template <int D, int MR>
hipError_t launch_tok_d(int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    switch (flags) {
        // MXFP8 (no dilated convolutions)
        case TOK_MX | TOK_EMBED | TOK_QKV: launch_variant<D, MR, TOK_MX | TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_MX | TOK_POST | TOK_QKV: launch_variant<D, MR, TOK_MX | TOK_POST | TOK_QKV>(p, n_tb, s); break;
        case TOK_MX | TOK_POST | TOK_EMBED | TOK_QKV:
            launch_variant<D, MR, TOK_MX | TOK_POST | TOK_EMBED | TOK_QKV>(p, n_tb, s);
            break;
        case TOK_MX | TOK_POST: launch_variant<D, MR, TOK_MX | TOK_POST>(p, n_tb, s); break;
        case TOK_MX | TOK_EMBED | TOK_QKV | TOK_RESNET:
            launch_variant<D, MR, TOK_MX | TOK_EMBED | TOK_QKV | TOK_RESNET>(p, n_tb, s);
            break;
        case TOK_MX | TOK_POST | TOK_EMBED | TOK_QKV | TOK_RESNET:
            launch_variant<D, MR, TOK_MX | TOK_POST | TOK_EMBED | TOK_QKV | TOK_RESNET>(p, n_tb, s);
            break;
        case TOK_EMBED | TOK_QKV: launch_variant<D, MR, TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST | TOK_QKV: launch_variant<D, MR, TOK_POST | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST | TOK_EMBED | TOK_QKV: launch_variant<D, MR, TOK_POST | TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_POST: launch_variant<D, MR, TOK_POST>(p, n_tb, s); break;
        case TOK_EMBED | TOK_QKV | TOK_RESNET: launch_variant<D, MR, TOK_EMBED | TOK_QKV | TOK_RESNET>(p, n_tb, s); break;
        case TOK_POST | TOK_EMBED | TOK_QKV | TOK_RESNET:
            launch_variant<D, MR, TOK_POST | TOK_EMBED | TOK_QKV | TOK_RESNET>(p, n_tb, s);
            break;
        // split POST around the dilated convolutions
        case TOK_WO: launch_variant<D, MR, TOK_WO>(p, n_tb, s); break;
        case TOK_FFN | TOK_QKV: launch_variant<D, MR, TOK_FFN | TOK_QKV>(p, n_tb, s); break;
        case TOK_FFN | TOK_EMBED | TOK_QKV: launch_variant<D, MR, TOK_FFN | TOK_EMBED | TOK_QKV>(p, n_tb, s); break;
        case TOK_FFN | TOK_EMBED | TOK_QKV | TOK_RESNET:
            launch_variant<D, MR, TOK_FFN | TOK_EMBED | TOK_QKV | TOK_RESNET>(p, n_tb, s);
            break;
        case TOK_FFN: launch_variant<D, MR, TOK_FFN>(p, n_tb, s); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// One residual unit of the dilated convolutions (model table: 3 x Conv2d(D, D) per layer;
// App. A.2: the attention output scattered onto the 2-D grid), an implicit GEMM on MFMA:
//   X[tok] += ReLU(b + sum_{a,e} W[a][e]^T G[cell(tok) + dil (a-1, e-1)])   (zero off the grid)
// Same structure as the token kernel's out-projection: 2 16-token blocks per wavefront, the
// accumulators (tokens along MFMA columns) in registers across all 9 taps, and the weights of
// each tap streamed through the double-buffered LDS ring. At each tap the wavefront gathers
// the B fragments of its tokens' neighbours (16 bytes per lane and k-step from the token-major
// bf16 copy G, which stays in L2), so every gathered fragment feeds D/16 MFMAs and every LDS
// weight fragment 2 per wavefront. Where registers allow (D = 128) the gathers run two taps
// ahead (see below). The residual stream stays fp32; the unit also writes its output as the
// next unit's G.
template <int D, bool GOUT>
__global__ __launch_bounds__(256, 2) void conv_kernel(ConvParams p) {
    constexpr int WAVES = 4;
    using S = Shape<D, WAVES, 4>;
    constexpr int RT = S::RT, KS = S::KS, CHUNK = S::CHUNK, LA = TOK_LA_WO;
    constexpr int TAP_CHUNKS = RT * KS / CHUNK;   // 4 at D = 256, 1 at D = 128
    static_assert(RT * KS % CHUNK == 0, "whole chunks per tap");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, col = lane & 15;
    // XCD-aware tiles: workgroups are dispatched round-robin over the 8 XCDs, so workgroup i
    // takes tile (i % 8) * (grid / 8) + i / 8 and each XCD sweeps a contiguous run of tiles,
    // whose neighbour gathers then share that XCD's L2. The grid is padded to a multiple of 8;
    // a workgroup past the last tile leaves before touching memory.
    const int n_wg = (int)(((int64_t)p.nwin * p.nbw + WAVES * TB - 1) / (WAVES * TB));
    const int per_xcd = (int)gridDim.x / 8;
    const int wg = (int)(blockIdx.x % 8) * per_xcd + (int)(blockIdx.x / 8);
    if (wg >= n_wg) return;
    const int64_t tb0 = ((int64_t)wg * WAVES + wave) * TB;

    WeightPipe<CHUNK, WAVES> pipe;
    pipe.post = p.stream;
    pipe.qkv = p.stream;
    pipe.n_post = 9 * TAP_CHUNKS;
    pipe.total = 9 * TAP_CHUNKS;
    pipe.wave = __builtin_amdgcn_readfirstlane(wave);
    pipe.lane = lane;

    f32x4 acc[RT][TB];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const f32x4 bias = ld4(p.bias + rt * 16 + 4 * g);
#pragma unroll
        for (int b = 0; b < TB; ++b) acc[rt][b] = bias;
    }
    pipe.template issue<0>(0);

    // this lane's token in each block: its cell and its window's first token
    const int side = p.d + 1;
    int r0[TB], c0[TB];
    bool real[TB];
    int64_t tok0[TB];
#pragma unroll
    for (int b = 0; b < TB; ++b) {
        const int64_t tb = tb0 + b;
        const int64_t w = tb / p.nbw;
        const int s = (int)(tb - w * p.nbw) * 16 + col;
        real[b] = w < p.nwin && s < p.ntok;
        r0[b] = s / side;
        c0[b] = s - r0[b] * side;
        tok0[b] = w * p.nbw * 16;
    }
    // D = 128: the gathers run two taps ahead in three register slots (tap t in slot t % 3),
    // each issued right after the last weight load of the chunk two taps earlier, so a chunk
    // sync need not wait for the newest gathers: vector memory completes in issue order, and
    // waiting until KS * TB operations remain leaves exactly those. D = 256: one slot,
    // gathered at the tap (no registers for more).
    constexpr int NSLOT = D <= 128 ? 3 : 1;
    bf16x8 xb[NSLOT][KS][TB];
    // the neighbours' B fragments for tap (a, e) = (tap / 3, tap % 3) into slot SLOT; every
    // load is issued, and an off-grid neighbour reads a row of zeros, so the loaded values
    // need no fix-up (which the compiler would schedule ahead, waiting on the prefetch early)
    auto gather = [&](auto slot, int tap) {
        constexpr int SLOT = decltype(slot)::value;
        const int dr = p.dil * (tap / 3 - 1), dc = p.dil * (tap % 3 - 1);
#pragma unroll
        for (int b = 0; b < TB; ++b) {
            const int rr = r0[b] + dr, cc = c0[b] + dc;
            const bool ok = real[b] && rr >= 0 && rr < side && cc >= 0 && cc < side;
            const uint16_t* src = (ok ? p.Gin + (tok0[b] + rr * side + cc) * KS * 32 : p.zero) + g * 8;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                xb[SLOT][ks][b] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(src + ks * 32));
        }
    };
    // chunk C of a tap (fragments C*CHUNK .. of the tap's [row tile][k-step] order) on the
    // gathered fragments in slot SLOT. YOUNGER: vector memory operations issued after this
    // chunk's last weight load (prefetched gathers); extra(r) runs after fragment read r.
    auto chunk = [&](auto par, auto cidx, auto slot, auto younger, int ci, const auto& extra) {
        constexpr int PAR = decltype(par)::value, C = decltype(cidx)::value, SLOT = decltype(slot)::value;
        const uint16_t* buf = pipe.template sync<PAR, decltype(younger)::value>(ci);
        const uint16_t* nx = pipe.next(ci);
        pipelined<CHUNK, LA>(
            [&](int r) { return lds_frag(buf, r, lane); },
            [&](int r, const bf16x8& a) {
                const int fr = C * CHUNK + r, rt = fr / KS, ks = fr % KS;
#pragma unroll
                for (int b = 0; b < TB; ++b) acc[rt][b] = mfma16x16x32(a, xb[SLOT][ks][b], acc[rt][b]);
            },
            [&](int r) {
                pipe.template after_read<1 - PAR, CHUNK, LA>(nx, r);
                extra(r);
            });
        sched_pipeline<CHUNK, TB, LA>();
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // the residual X of the workgroup's tokens, loaded during the last tap (D = 128: into the
    // registers the first two gather slots free by then) or at the end
    f32x4 xold[RT][TB];
    auto load_x = [&]() {
#pragma unroll
        for (int b = 0; b < TB; ++b)
#pragma unroll
            for (int rt = 0; rt < RT; ++rt)
                xold[rt][b] = ld_stream(reinterpret_cast<const f32x4*>(p.X + (((tb0 + b) * RT + rt) * 64 + lane) * 4));
    };
    if constexpr (NSLOT == 3) {
        static_assert(TAP_CHUNKS == 1, "one chunk per tap");
        constexpr int LAST = WeightPipe<CHUNK, WAVES>::template last_load_read<CHUNK, LA>();
        gather(I0{}, 0);
        gather(I1{}, 1);
        static_for<9>([&](auto tc) {
            constexpr int T = decltype(tc)::value;
            // at chunk T's sync, tap T + 1's gathers (issued after chunk T - 1's last weight
            // load, or after chunk 0's first loads in the prologue) may still be in flight
            constexpr int YOUNGER = T + 1 < 9 ? KS * TB : 0;
            chunk(std::integral_constant<int, T & 1>{}, I0{}, std::integral_constant<int, T % 3>{},
                  std::integral_constant<int, YOUNGER>{}, T, [&](int r) {
                      if constexpr (T + 2 < 9)
                          if (r == LAST) gather(std::integral_constant<int, (T + 2) % 3>{}, T + 2);
                      if constexpr (T == 8)
                          if (r == 0) load_x();   // after the last sync: no chunk waits for these
                  });
        });
    } else {
        static_assert(TAP_CHUNKS % 2 == 0, "chunk parity is the chunk's index within its tap");
        for (int tap = 0; tap < 9; ++tap) {
            gather(I0{}, tap);
            static_for<TAP_CHUNKS>([&](auto c) {
                constexpr int C = decltype(c)::value;
                chunk(std::integral_constant<int, C & 1>{}, c, I0{}, I0{}, tap * TAP_CHUNKS + C, [](int) {});
            });
        }
        load_x();
    }

    // X += ReLU(acc); the output's B fragments for the next unit
#pragma unroll
    for (int b = 0; b < TB; ++b)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            f32x4 xo[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                f32x4* px = reinterpret_cast<f32x4*>(p.X + (((tb0 + b) * RT + 2 * ks + h) * 64 + lane) * 4);
                xo[h] = xold[2 * ks + h][b] + relu4(acc[2 * ks + h][b]);
                st_stream(px, xo[h]);
            }
            if constexpr (GOUT)
                st_l2(reinterpret_cast<u16x8*>(p.Gout + ((((tb0 + b) * 16 + col) * KS + ks) * 4 + g) * 8),
                          __builtin_bit_cast(u16x8, pack_b(xo[0], xo[1])));
        }
    // the last chunk's reload into the idle buffer lands before the LDS is freed
    constexpr int END_YOUNGER = RT * TB + (GOUT ? KS * TB : 0);
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(END_YOUNGER) : "memory");
}

}  // namespace

hipError_t launch_conv(int D, bool gout, const ConvParams& p, int64_t n_tb, hipStream_t s) {
    if (n_tb <= 0) return hipSuccess;
    // the kernel maps workgroups to tiles XCD by XCD: the grid is padded to a multiple of 8
    const int64_t n_wg = (n_tb + 4 * TB - 1) / (4 * TB);
    const dim3 grid((unsigned)((n_wg + 7) / 8 * 8)), block(256);
    if (D == 256 && gout) conv_kernel<256, true><<<grid, block, 0, s>>>(p);
    else if (D == 256) conv_kernel<256, false><<<grid, block, 0, s>>>(p);
    else if (D == 128 && gout) conv_kernel<128, true><<<grid, block, 0, s>>>(p);
    else if (D == 128) conv_kernel<128, false><<<grid, block, 0, s>>>(p);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// Token blocks are processed in groups of 8 or 16 (wavefronts x TB by variant); every buffer
// indexed here must be allocated for n_tb rounded up to a multiple of all of them.
int64_t tok_block_granule() { return 48; }

// Fragments of the weight streams (see tok_kernel): hidden units per feed-forward chunk.
int tok_mlp_chunk(int D) { return 8192 / D; }

// Copies of each V bias value in the Q/K/V bias table: [b_q b_k] then b_v, each value rep times.
int tok_bv_rep(int D, int F) { return bv_rep(D, F); }

int tok_mx_qkv_frags() { return Shape<256, 4, 4>::MX_QKV_FRAGS; }
int tok_mx_scale_slot() { return Shape<256, 4, 4>::MX_SCALE_SLOT; }

hipError_t launch_tok(int D, int F, int flags, const TokParams& p, int64_t n_tb, hipStream_t s) {
    if (n_tb <= 0) return hipSuccess;
    if (D == 256 && F == 4 * D) return launch_tok_d<256, 4>(flags, p, n_tb, s);
    if (D == 256 && F == 5 * D) return launch_tok_d<256, 5>(flags, p, n_tb, s);
    if (D == 128 && F == 4 * D) return launch_tok_d<128, 4>(flags, p, n_tb, s);
    if (D == 128 && F == 5 * D) return launch_tok_d<128, 5>(flags, p, n_tb, s);
    return hipErrorInvalidValue;
}
