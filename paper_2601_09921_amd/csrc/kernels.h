// Kernel parameter blocks and launchers of the decoder (host <-> device interface inside
// the library; nothing here is part of the public C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

// Window geometry and input pointers common to the stages that read syndromes.
struct SyndromeIn {
    const uint32_t* meas;   // [nwin][W+1][words]
    const uint8_t* types;   // [nwin]
    int nwin, W, words, d, N, b_left;
};

// Stage flags of the token-local kernel.
// POST = out-projection + LN1 + feed-forward + LN2. With the dilated convolutions between LN1
// and the feed-forward, POST splits into WO (out-projection + LN1, alone; also writes the
// convolutions' bf16 input G) and FFN (feed-forward + LN2, then EMBED / QKV as after POST).
// MX: the Q/K/V projections and the feed-forward's first matrix take MXFP8 operands (E4M3
// elements, one E8M0 scale per 32-feature block; see tok.hip); their weight streams are laid
// out for it.
enum { TOK_POST = 1, TOK_EMBED = 2, TOK_QKV = 4, TOK_RESNET = 8, TOK_WO = 16, TOK_FFN = 32, TOK_MX = 64 };

struct TokParams {
    SyndromeIn in;          // in.N: stabilizers (bits per measurement round)
    int ntok;               // tokens per window (in.N, or (d+1)^2 for the grid token set)
    const int* tok_stab;    // [ntok] stabilizer of each token or -1; null: token s = stabilizer s
    int Npad, nbw;          // padded tokens and 16-token blocks per window
    int t;                  // round whose embedding TOK_EMBED adds
    float kappa, eps;
    float qscale;           // log2(e)/sqrt(dh): Q is stored pre-scaled for exp2-based softmax
    float* X;               // fp32 residual / state, C fragments
    uint16_t* QKV;          // bf16 B fragments [tb][3][D/32][64][8]
    const uint16_t* Y;      // bf16 attention output [tb][D/32][64][8]
    const float* S0;        // b_e + PE, fp32 C fragments [nbw][D/16][64][4] (0 on padding)
    const float* we;        // [D]
    // weight streams: bf16 A fragments in consumption order (see tok.hip)
    const uint16_t* post_stream;   // out-projection + feed-forward of the POST layer
    const uint16_t* qkv_stream;    // Q/K/V projection of the layer that follows
    const float* post_vecs;   // POST layer vectors [b_o g1 be1 b2 g2 be2 | b1], 10 D floats
    const float* bqkv;      // [6D] bias of the Q/K/V projection: b_q, b_k, then b_v with each value x 4
    uint16_t* state_out;    // POST|EMBED: if not null, D_t (before the fold) as bf16 C fragments
    // TOK_RESNET: the embedder's residual Conv1d block as a lookup (see pwdec.cpp)
    const int* emb_nb;      // [ntok][8]: stabilizers at cells c-2 .. c+2 of the token's cell c
                            // (-1: none), then the cell's position class (0..4), 0, 0
    const float* emb_tab;   // [5 * 32][D]: block output by (position class, 5 event bits)
    uint16_t* G;            // TOK_WO: the LN1 output as bf16 B fragments, token-major
                            // [tb * 16 + col][D/32][4][8] (k-step, lane group, 8 values)
};

// One residual unit of the dilated convolutions on the (d+1)^2 grid (the grid token set: token
// = cell r*(d+1)+c): X = X + ReLU(b + sum_taps W_tap^T x[cell + dil * offset]).
struct ConvParams {
    float* X;               // fp32 state, C fragments [tb][D/16][64][4]: residual in, result out
    const uint16_t* Gin;    // the unit's input as bf16 B fragments, token-major (TokParams::G)
    uint16_t* Gout;         // its output in the same layout (the next unit's input)
    const uint16_t* stream; // weight fragments: 9 taps (3 a + e) x [D/16 row tiles][D/32 k-steps]
    const float* bias;      // [D]
    const uint16_t* zero;   // D zero values: what an off-grid neighbour reads
    int d, dil, ntok, nbw, nwin;
};

struct AttnParams {
    const uint16_t* QKV;
    uint16_t* Y;
    int N, Npad, nbw, H;    // Q arrives pre-scaled by log2(e)/sqrt(dh)
};

struct ReadoutParams {
    const float* X;         // decoder state, fp32 C fragments [tb][D/16][64][4] ...
    const uint16_t* Xb;     // ... or, when not null, the same layout in bf16
    const uint8_t* types;
    float* logits;          // logits[win * stride]
    uint8_t* bits;          // bits[win * stride]
    int stride;
    int* err;               // device error word
    const uint16_t* Wc;     // bf16 A fragments of Wc^T: [D/16][4D/32][64][8], k = tap*D + in
    const float* bc;        // [D]
    const float* wo;        // [d][D]
    float bo;
    float beta[3];
    const int* cell_token;  // [(d+1)*(d+1)] token index or -1
    int nwin, d, D, nbw;
};

struct EventsParams {
    SyndromeIn in;
    uint32_t* events;       // [nwin][W][words]
    int* err;
};

struct F32Params {
    SyndromeIn in;          // in.N: stabilizers (bits per measurement round)
    int ntok;               // tokens per window
    const int* tok_stab;    // [ntok] stabilizer of each token or -1; null: token s = stabilizer s
    const float* w;         // blob tensors in blob order (fp32)
    const float* S0;        // b_e + PE per token [ntok][D]
    const int* cell_token;  // [(d+1)*(d+1)]
    float* logits;          // logits[win * readouts + k] after round W - readouts + k
    uint8_t* bits;
    int* err;
    int D, L, H, F;
    const int* emb_nb;      // embedder residual block as in TokParams, or null
    const float* emb_tab;
    const float* conv_w;    // dilated convolutions: per layer Wd[3][3][3][D][D] bd[3][D], or null
    int dil[3];             // their dilations (grid token set: token = cell)
    int readouts;           // readouts after the last `readouts` rounds (1: final state only)
    float kappa, eps;
};

// The state-resident decoder (resident.hip): every round and layer of a batch of windows in
// one launch, one wavefront per window, the state in registers. It writes the final state
// D_W to X for the readout.
struct ResidentParams {
    SyndromeIn in;
    int ntok;               // tokens per window
    const int* tok_stab;    // [ntok] stabilizer of each token or -1; null: token s = stabilizer s
    int nbw;                // 16-token blocks per window (1..4)
    int L;                  // layers
    float kappa, eps, qscale;
    const uint16_t* stream; // weight fragments of every layer in consumption order (see resident.hip)
    const float* vecs;      // [L][9 D + F]: b_q b_k b_v b_o g1 be1 b2 g2 be2 b1
    const float* S0;        // b_e + PE, fp32 C fragments [nbw][D/16][64][4]
    const float* we;        // [D]
    float* X;               // out: the final state, fp32 C fragments [nwin * nbw][D/16][64][4]
};
bool resident_supported(int D, int nbw, int L, int mr, int dh);
int resident_chunk_fragments();
hipError_t launch_resident(int mr, int dh, const ResidentParams& p, hipStream_t s);

hipError_t launch_events(const EventsParams& p, hipStream_t s);
int64_t tok_block_granule();
int tok_mlp_chunk(int D);
int tok_bv_rep(int D, int F);
int tok_mx_qkv_frags();     // MXFP8 fragments per Q/K/V chunk
int tok_mx_scale_slot();    // 1 KB slot of a chunk that holds its MXFP8 weight scales
hipError_t launch_tok(int D, int F, int flags, const TokParams& p, int64_t n_tb, hipStream_t s);
hipError_t launch_conv(int D, bool gout, const ConvParams& p, int64_t n_tb, hipStream_t s);
hipError_t launch_attn(int dh, const AttnParams& p, int nwin, hipStream_t s);
hipError_t launch_readout(const ReadoutParams& p, hipStream_t s);
hipError_t launch_f32_window(const F32Params& p, hipStream_t s);
size_t f32_window_smem_bytes(int N, int D, int H, int F);
size_t attn_smem_bytes(int dh, int Npad, int nbw);

// Stream decoding (stream.hip)
struct StreamSplitParams {
    const uint32_t* stream;   // [T][words]
    int64_t T;
    int m, d, W, b_left, words;
    uint32_t* meas;           // [m][W + 1][words] out
    uint8_t* types;           // [m] out
};
struct StreamCombineParams {
    const float* logits;      // [m]
    const uint8_t* bits;      // [m]
    int m;
    uint8_t* bit;             // [1] out
    float* prob;              // [1] out, or null
    float* probs;             // [m] out, or null: sigmoid of each window's logit
};
hipError_t launch_stream_split(const StreamSplitParams& p, hipStream_t s);
hipError_t launch_stream_combine(const StreamCombineParams& p, hipStream_t s);
