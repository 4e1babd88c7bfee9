/*
 * pwdec.h - C ABI of the MI355X parallel-window neural decoder.
 *
 * The library decodes many independent decoding windows of a distance-d rotated surface
 * code in parallel. Each window takes the syndromes of its rounds and outputs one logit
 * and one correction bit for its core region (Sec. 3.1; Algorithm 1, inference branch,
 * with the input of shape batch x rounds x stabilizers). The per-window bits of a memory
 * experiment combine by XOR into the global logical correction (eq. global_xor).
 *
 * Conventions shared by every entry point:
 *  - Every function returns PWD_OK (0) on success or a negative pwd_status. No C++
 *    exception crosses the ABI. On failure decoder_last_error() describes the cause.
 *  - Pointers named d_* are device pointers (HIP global memory of the decoder's device);
 *    the caller owns and allocates them. Host pointers are read during the call only.
 *  - hip_stream is a hipStream_t (NULL = the default stream). Device work is enqueued on
 *    it and the call returns without synchronising; results are valid once the stream
 *    has been synchronised. A handle holds scratch memory sized for max_windows, so one
 *    handle must not run on two streams at once.
 *  - Stabilizer bits are packed LSB-first into uint32 words: the bit of stabilizer s is
 *    bit (s % 32) of word (s / 32); words = ceil((d*d-1)/32). Input bits at positions
 *    >= d*d-1 are ignored; output bits there are written as 0.
 *  - Stabilizer (token) order: the d*d-1 stabilizers of the rotated surface code in
 *    row-major order of their cell (r, c) on the (d+1)x(d+1) lattice (App. A.1.2). A
 *    stabilizer at (r, c) acts on data qubits (r-1..r, c-1..c) inside the d x d patch;
 *    interior cells 1 <= r, c <= d-1 are weight 4, top/bottom edge cells are kept when
 *    r+c is even, left/right edge cells when r+c is odd.
 */
#ifndef PWDEC_H
#define PWDEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pwd_decoder pwd_decoder; /* opaque handle */

/* Window geometry (Sec. 3.1, App. A.1.1 boundary padding, App. A.1.2: a window is b + c + b
 * rounds). A window has window_rounds rounds: a left buffer of
 * floor((window_rounds - distance) / 2) rounds, a core of `distance` rounds and a right
 * buffer of the rest. There is no separate core-length field: the core length c always
 * equals the code distance (the paper's windows take c = d; every window of a stream then
 * owns exactly d rounds, App. A.1.1), so the geometry is fixed by distance and
 * window_rounds alone. distance: odd, 3..63 within the on-chip limits that
 * decoder_validate_config states (bf16: up to 35). window_rounds: distance..3*distance (the
 * paper's b = c = d is window_rounds = 3*distance). max_windows: the largest batch
 * decode_windows will be given (scratch is sized for it). */
typedef struct {
    int32_t distance;
    int32_t window_rounds;
    int32_t max_windows;
} pwd_geometry;

/* Network dimensions (App. A model table): d_model, layers, heads, MLP expansion (the
 * feed-forward width is mlp_ratio * d_model; the model table gives 5), the arithmetic type,
 * the token set, the embedder and the dilated convolutions (see the enums below).
 * PWD_DTYPE_BF16: bf16 weights and matrix operands, fp32 accumulation, softmax, LayerNorm,
 * residual stream and recurrent state. PWD_DTYPE_F32: fp32 throughout. PWD_DTYPE_MXFP8: as
 * bf16, except that the Q, K and V projections and the feed-forward's first matrix (d_model ->
 * F) of every layer take MXFP8 operands (quantization, named in Sec. 1 and Sec. 5 as the route
 * toward the real-time budget): OCP Microscaling v1.0 FP8 E4M3 elements with one E8M0 scale
 * 2^(floor(log2 amax) - 8) per block of 32 input features (each 128-feature slice splits into
 * four blocks; feature f is in block 4 (f/128) + 2 ((f/64) % 2) + (f/8) % 2), elements rounded
 * to nearest even and clamped to +-448; one scale per token and block for the activations
 * (quantized on the fly), one per output feature and block for the weights (quantized once,
 * by decoder_create); fp32 accumulation. PWD_TOKENS_STABILIZERS: one token per stabilizer (d*d-1); PWD_TOKENS_GRID: one
 * token per cell of the (d+1)x(d+1) stabilizer array (App. A.1.2 and the (d+1)^2 x d_model
 * state of Algorithm 1), the cells without a stabilizer carrying state but no detection
 * events. Syndrome inputs and detection events stay one bit per stabilizer either way. */
typedef struct {
    int32_t d_model;
    int32_t n_layers;
    int32_t n_heads;
    int32_t mlp_ratio;
    int32_t dtype;
    int32_t token_set;
    int32_t embedder;
    int32_t conv_dilation[3];
} pwd_model_dims;

enum { PWD_DTYPE_F32 = 0, PWD_DTYPE_BF16 = 1, PWD_DTYPE_MXFP8 = 2 };
enum { PWD_TOKENS_STABILIZERS = 0, PWD_TOKENS_GRID = 1 };
/* PWD_EMBED_LINEAR: the embedding is Linear(1 -> d_model) of each event bit plus PE.
 * PWD_EMBED_RESNET: the model table's StabilizerEmbedder, Linear(1 -> d_model) followed by a
 * residual block of two Conv1d(d_model, d_model) layers along the flattened (d+1)x(d+1)
 * stabilizer array, ahead of PE (syndrome-convolution section): with E the Linear output at
 * every cell (e = 0 at cells without a stabilizer), E + Conv2(ReLU(Conv1(E))), kernel 3,
 * zero padding 1, biases. */
enum { PWD_EMBED_LINEAR = 0, PWD_EMBED_RESNET = 1 };
/* conv_dilation: all zero, or the dilations (1..distance) of the Syndrome Transformer's three
 * dilated convolutions (model table: 3 x Conv2d(d_model, d_model); App. A.2: the attention
 * output scattered onto the 2-D grid). Each layer then runs, between LayerNorm 1 and the
 * feed-forward, three residual units C = C + ReLU(b_j + Conv2d_j(C)) with 3x3 kernels,
 * dilation conv_dilation[j] and zero padding equal to it, over the (d+1)x(d+1) grid. They
 * need the PWD_TOKENS_GRID token set (every cell a token). */

/* Window types (App. A.1.1): the initial window has zero padding in place of its left
 * buffer, the final window in place of its right buffer. */
enum { PWD_WIN_INITIAL = 0, PWD_WIN_BULK = 1, PWD_WIN_FINAL = 2 };

typedef enum {
    PWD_OK = 0,
    PWD_EINVAL = -1,       /* null pointer, negative size or malformed argument */
    PWD_EUNSUPPORTED = -2, /* geometry or dimensions outside the supported range */
    PWD_EBLOB = -3,        /* weight blob: bad magic, version, size or header mismatch */
    PWD_ENOMEM = -4,       /* device or host allocation failed */
    PWD_EHIP = -5,         /* a HIP runtime call failed (message in decoder_last_error) */
    PWD_EBATCH = -6,       /* n_windows > max_windows */
    PWD_EDEVICE = -7       /* a device-side check fired (an invalid window type) */
} pwd_status;

/* Weight blob, version 1. All fields little-endian.
 *   header: 16 x 32-bit words
 *     [0] magic 0x31445750 ("PWD1")  [1] version = 1
 *     [2] distance  [3] window_rounds  [4] d_model  [5] n_layers  [6] n_heads
 *     [7] mlp hidden size F = mlp_ratio * d_model  [8] dtype
 *     [9] fold constant kappa (float32 bits; App. A.2 uses 0.707)
 *     [10] LayerNorm epsilon (float32 bits)  [11] token set  [12] embedder
 *     [13] conv dilations, byte j = conv_dilation[j]  [14..15] zero
 *   then float32 tensors, row-major, matrices stored [in][out] (y = x W + b):
 *     w_e[D], b_e[D]                                    StabilizerEmbedder Linear(1 -> D)
 *     per layer: Wq[D][D] bq[D] Wk[D][D] bk[D] Wv[D][D] bv[D] Wo[D][D] bo[D]
 *                g1[D] be1[D] W1[D][F] b1[F] W2[F][D] b2[D] g2[D] be2[D]
 *     Wc[2][2][D][D] bc[D]                              readout 2x2 convolution
 *     w_o[d][D] b_o[1]                                  readout Linear(d*D -> 1)
 *     beta[3]                                           logit bias per window type
 *     PWD_EMBED_RESNET only: Wr1[3][D][D] br1[D] Wr2[3][D][D] br2[D]   the two Conv1d layers,
 *                                                       weights [tap][in][out], tap k reading
 *                                                       the cell at offset k - 1
 *     dilated convolutions only, per layer: Wd[3][3][3][D][D] bd[3][D]   ([j][a][e][in][out]:
 *                                                       unit j, tap (a, e) reading the cell
 *                                                       at dil_j (a - 1, e - 1))
 * For PWD_DTYPE_BF16 and PWD_DTYPE_MXFP8 the values are used rounded to bf16, those of Wq, Wk,
 * Wv and W1 under MXFP8 quantized from the given float32 values instead (they should already be
 * bf16-representable). The positional encoding is not stored: the library computes it. */
#define PWD_BLOB_MAGIC 0x31445750u
#define PWD_BLOB_VERSION 1
#define PWD_BLOB_HEADER_WORDS 16

/* Number of float32 values that follow the blob header for these dimensions. */
size_t decoder_blob_floats(const pwd_geometry* geom, const pwd_model_dims* dims);

/* Checks geometry and dimensions on the host only; touches no device.
 * Supported: distance odd in 3..63 with the on-chip limits below (bf16: up to 35 at head
 * sizes 16 and 32, up to 25 at 64); distance <= window_rounds <= 3*distance;
 * 1 <= max_windows <= 2^24; mlp_ratio 4 or 5; n_layers 1..8;
 * token_set PWD_TOKENS_STABILIZERS or PWD_TOKENS_GRID (n_tokens = d*d-1 or (d+1)^2);
 * embedder PWD_EMBED_LINEAR or PWD_EMBED_RESNET; conv_dilation all 0, or all in 1..distance
 * with PWD_TOKENS_GRID;
 * PWD_DTYPE_MXFP8: as PWD_DTYPE_BF16, without the dilated convolutions;
 * PWD_DTYPE_BF16: d_model in {128, 256}, head size d_model/n_heads in {16, 32, 64}, and the
 * attention tile (K and V of one head: (2 ceil(n_tokens/16) + 1) KB, twice that for head size
 * 64) within 160 KB of LDS;
 * PWD_DTYPE_F32: d_model in {16, 32, 64}, head size in {4, 8, 16, 32, 64} and the window
 * (n_tokens * (6 d_model + F) + n_heads * n_tokens^2) * 4 bytes within 64 KB of LDS (about
 * d <= 5 at d_model 64). Returns PWD_OK, PWD_EINVAL (null) or PWD_EUNSUPPORTED. */
int decoder_validate_config(const pwd_geometry* geom, const pwd_model_dims* dims);

/* Creates a decoder on the current HIP device. The blob carries the parameters of the
 * network of the App. A model table (StabilizerEmbedder Linear(1 -> d_model), the Syndrome
 * Transformer layers of App. A.2 with the fold of the recurrent state, the readout of
 * App. A.3) in the order listed above; decoder_create validates the dimensions, parses the
 * blob (blob_bytes must equal 64 + 4 * decoder_blob_floats; PWD_EBLOB on a bad magic,
 * version, size or a header word that disagrees with geom / dims), computes the
 * positional encoding of App. A.1.4 on the host, rearranges the weights into the kernels'
 * layouts, uploads them and allocates scratch for max_windows windows (PWD_ENOMEM if the
 * device allocation fails). The caller keeps ownership of weight_blob and may free it on
 * return; the handle owns its device memory until decoder_destroy. *out is set only on
 * success. */
int decoder_create(const pwd_geometry* geom, const pwd_model_dims* dims,
                   const void* weight_blob, size_t blob_bytes, pwd_decoder** out);

/* Decodes n_windows windows (Algorithm 1, inference branch, then the readout of App. A.3).
 *   d_meas:   uint32 [n_windows][window_rounds + 1][words] stabilizer measurements; row 0
 *             is the round just before the window's first round. Detection events are
 *             E[t] = M[t+1] xor M[t]; an initial window zeroes E[t] for t < left buffer
 *             and compares its first core round with the all-zero state; a final window
 *             zeroes E[t] from the end of its core on.
 *   d_types:  uint8 [n_windows], each PWD_WIN_INITIAL / BULK / FINAL.
 *   d_logits: float [n_windows] out; d_bits: uint8 [n_windows] out, 1 iff logit > 0.
 * n_windows = 0 is a no-op. A window with type > 2 gets logit NaN, bit 0, and makes the
 * next decoder_sync_status return PWD_EDEVICE. Results do not depend on the batch size
 * or on a window's position in the batch. */
int decode_windows(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types,
                   int64_t n_windows, float* d_logits, uint8_t* d_bits, void* hip_stream);

/* Bytes of device scratch that decode_windows_noalloc can use on each GPU (see there). */
#define PWD_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* For callers that cannot allocate device memory at call time or hold a per-handle workspace
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * decode_windows with its activations (fp32 state, Q/K/V, attention output, and the two
 * convolution buffers with dilated convolutions) in a fixed array of PWD_NOALLOC_SCRATCH_BYTES
 * that the library reserves in device memory when it is loaded, instead of the handle's
 * scratch. Arguments, outputs, results and errors as for decode_windows; it calls no hipMalloc,
 * hipFree or other allocating routine. The bf16 path needs
 *   (48 * ceil(n_windows * ceil(n_tokens / 16) / 48) * 16 * d_model * 12 bytes
 * (18 per token and feature with dilated convolutions), at most PWD_NOALLOC_SCRATCH_BYTES, e.g.
 * up to 68 windows at d = 25 with d_model 256 and 1808 at d = 7 with d_model 128; a larger batch
 * returns PWD_EBATCH and launches nothing. The fp32 path keeps each window on chip and uses none.
 * The array is one per GPU and shared by every call and every handle on that GPU, so calls that
 * overlap on one GPU (two streams, two threads) race and must be serialised by the caller. It
 * keeps the previous call's contents; no part of it needs to start at any particular value
 * (every element a decode reads is written earlier in the same decode, except padding blocks
 * past the batch, whose results are discarded). */
int decode_windows_noalloc(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types,
                           int64_t n_windows, float* d_logits, uint8_t* d_bits, void* hip_stream);

/* The recurrent branch of Algorithm 1 (Sec. recurrent training): the same pass over each
 * window, with a readout of the decoder state after every round n > W - distance (the rounds
 * that complete a window of left buffer, tau core and right buffer rounds, tau = 1..distance).
 *   d_logits: float [n_windows][distance] out, column tau-1 after round W - distance + tau;
 *   d_bits:   uint8 [n_windows][distance] out, 1 iff logit > 0.
 * The last column is what decode_windows returns. Arguments, errors and the type check as
 * for decode_windows. */
int decode_windows_recurrent(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types,
                             int64_t n_windows, float* d_logits, uint8_t* d_bits, void* hip_stream);

/* Writes the detection events the decoder feeds to its network (Sec. 2.2: a detector is the
 * parity of two consecutive measurements of one stabilizer; Sec. 3.2: the model takes hard
 * detection events as its only input; App. A.1.1: zero padding in place of the missing
 * buffer of the initial and final windows):
 *   E[t] = M[t+1] xor M[t], t = 0 .. window_rounds - 1; an initial window zeroes E[t] for
 *   t < left buffer and compares its first core round with the all-zero state; a final
 *   window zeroes E[t] from the end of its core on.
 * d_meas and d_types as for decode_windows; d_events: uint32 [n_windows][window_rounds][words]
 * out (caller-allocated, device), packed as the input with bits >= d*d-1 written as 0. An
 * invalid type yields all-zero events for that window and makes the next
 * decoder_sync_status return PWD_EDEVICE. PWD_EINVAL on a null buffer or negative n,
 * PWD_EBATCH if n_windows > max_windows; n_windows = 0 is a no-op. */
int decoder_detection_events(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types,
                             int64_t n_windows, uint32_t* d_events, void* hip_stream);

/* Decodes a whole memory experiment (Sec. 3.1 windowing; eq. global_xor and eq. soft_xor).
 * The stream of T measurement rounds is cut on the device into m = ceil(T / distance)
 * windows: window i has core rounds [i d, i d + d) and rows R[i d - b_left - 1 + k] for
 * k = 0..window_rounds, b_left = (window_rounds - distance) / 2; rows before the stream read
 * as zeros and rows after it repeat round T-1 (the stream padded to m d rounds by holding its
 * last round). Window 0 is initial, window m-1 final, the others bulk. The windows are
 * decoded as by decode_windows and their results combined:
 *   d_stream:        uint32 [T][words] packed rounds, as the rows of decode_windows.
 *   d_window_logits: float [m] out, or NULL; d_window_bits: uint8 [m] out, or NULL.
 *   d_window_probs:  float [m] out, or NULL: each window's probability of a logical flip in its
 *                    core, y_k = 1 / (1 + exp(-logit_k)) (the sigmoid output the model is trained
 *                    on, Sec. 3.3; the inputs of eq. soft_xor), computed in double, rounded once.
 *   d_bit:           uint8 [1] out: XOR of the window bits, the global logical correction.
 *   d_prob:          float [1] out, or NULL: soft-XOR (1 - prod_k (1 - 2 y_k)) / 2 of the
 *                    window probabilities y_k, accumulated in double in a fixed order.
 * PWD_EINVAL if dec, d_stream or d_bit is NULL or T <= 0; PWD_EBATCH unless
 * 2 <= m <= max_windows. The window scratch (allocated by decoder_create) belongs to the
 * handle, so calls on one handle must not overlap. */
int decode_stream(pwd_decoder* dec, const uint32_t* d_stream, int64_t T, float* d_window_logits,
                  uint8_t* d_window_bits, float* d_window_probs, uint8_t* d_bit, float* d_prob, void* hip_stream);

/* Synchronises hip_stream, then reports PWD_EDEVICE if a device-side check fired since
 * the previous call (and clears it), PWD_EHIP on a stream error, else PWD_OK. */
int decoder_sync_status(pwd_decoder* dec, void* hip_stream);

/* Message of the last failure on the calling thread ("" if none). Valid until the next
 * call on this thread. */
const char* decoder_last_error(void);

/* Kernel stages of decode_windows, for per-stage timing. */
enum {
    PWD_STAGE_EMBED_QKV = 0,      /* round-0 embedding + layer-0 Q/K/V projection */
    PWD_STAGE_ATTENTION = 1,      /* multi-head self-attention, one launch per layer and round */
    PWD_STAGE_POST_QKV = 2,       /* out-projection, LayerNorms, feed-forward + next layer's Q/K/V */
    PWD_STAGE_POST_EMBED_QKV = 3, /* last layer of a round + next round's embedding and Q/K/V */
    PWD_STAGE_POST = 4,           /* last layer of the last round */
    PWD_STAGE_READOUT = 5,        /* readout */
    PWD_STAGE_FP32_WINDOW = 6,    /* the whole fp32 decoder (fp32 configurations) */
    PWD_STAGE_STREAM_SPLIT = 7,   /* decode_stream: cutting the stream into windows */
    PWD_STAGE_STREAM_COMBINE = 8, /* decode_stream: XOR and soft-XOR of the window results */
    PWD_STAGE_OUT_PROJ = 9,       /* with dilated convolutions: out-projection + LayerNorm 1
                                     (stages 2-4 then time the feed-forward part) */
    PWD_STAGE_DILATED_CONV = 10,  /* one launch per residual unit of the dilated convolutions */
    PWD_STAGE_RESIDENT = 11,      /* the state-resident schedule: every round and layer in one launch */
    PWD_NUM_STAGES = 12
};

/* Launch schedules of decode_windows (the network and its results are the same; Algorithm 1
 * carries the state D_n from round to round either way):
 *   PWD_SCHEDULE_LAYERS: one launch per layer and round for attention and one for the token-local
 *     stages, the state and activations of the whole batch in HBM between launches;
 *   PWD_SCHEDULE_RESIDENT: one launch for every round and layer, each window owned by one
 *     wavefront with its state, Q, K and V kept in registers throughout (PWD_DTYPE_BF16, d_model 128, at
 *     most 64 tokens and 4 layers, heads of 16 or 32, feed-forward 4 d_model, no dilated
 *     convolutions or embedder block), then the readout;
 *   PWD_SCHEDULE_AUTO (the default): RESIDENT where the configuration allows it, else LAYERS.
 * The recurrent branch (decode_windows_recurrent) always uses LAYERS. */
enum { PWD_SCHEDULE_AUTO = 0, PWD_SCHEDULE_LAYERS = 1, PWD_SCHEDULE_RESIDENT = 2 };

/* Selects the schedule of the handle's later decodes. PWD_EUNSUPPORTED if RESIDENT is asked for
 * a configuration outside its range, PWD_EINVAL for an unknown value. Host only. */
int decoder_schedule(pwd_decoder* dec, int schedule);

typedef struct {
    double ms[PWD_NUM_STAGES];       /* summed kernel time per stage, milliseconds */
    int64_t launches[PWD_NUM_STAGES];
} pwd_stage_times;

/* Turns per-stage kernel timing on (enable != 0) or off. While on, decode_windows records a
 * pair of HIP events around each kernel launch on its stream (no synchronisation inside the
 * call); the times accumulate until decoder_profile_read. Turning it on clears what was
 * accumulated. Costs one event record per launch. */
int decoder_profile(pwd_decoder* dec, int enable);

/* Synchronises the events recorded since the last read, adds their elapsed times to *out
 * (which the caller zeroes first) and releases them. PWD_EINVAL if out is NULL. */
int decoder_profile_read(pwd_decoder* dec, pwd_stage_times* out);

/* Frees the device memory of the handle. NULL is accepted. The caller must make sure no
 * work of this handle is still running. */
int decoder_destroy(pwd_decoder* dec);

#ifdef __cplusplus
}
#endif

#endif /* PWDEC_H */
