// Host side of the C ABI in include/pwdec.h: validation, weight-blob parsing, the rotated
// surface-code geometry, the positional-encoding table, weight relayout into MFMA
// fragments, device allocation and the per-round launch sequence (Algorithm 1).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/pwdec.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

#define HIP_OK(call)                                                                     \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess)                                                            \
            return fail(PWD_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));        \
    } while (0)

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceGuard(int dev) {
        err = hipGetDevice(&prev);
        if (err == hipSuccess && prev != dev) err = hipSetDevice(dev);
    }
    ~DeviceGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

uint16_t to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);   // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

int kslot(int g, int i) { return i < 4 ? 4 * g + i : 16 + 4 * g + (i - 4); }

// W is [K][O] row-major (y = x W). Output: A fragments of W^T, [O/16][K/32][64][8] bf16.
void append_frags(std::vector<uint16_t>& out, const float* W, int K, int O) {
    for (int ro = 0; ro < O / 16; ++ro)
        for (int ks = 0; ks < K / 32; ++ks)
            for (int lane = 0; lane < 64; ++lane)
                for (int i = 0; i < 8; ++i) {
                    const int row = ro * 16 + (lane & 15);
                    const int k = ks * 32 + kslot(lane >> 4, i);
                    out.push_back(to_bf16(W[(size_t)k * O + row]));
                }
}

// Stabilizer cells of the rotated surface code, row-major over the (d+1)x(d+1) lattice.
std::vector<std::pair<int, int>> stabilizer_cells(int d) {
    std::vector<std::pair<int, int>> cells;
    for (int r = 0; r <= d; ++r)
        for (int c = 0; c <= d; ++c) {
            const bool inner = r >= 1 && r <= d - 1 && c >= 1 && c <= d - 1;
            const bool tb = (r == 0 || r == d) && c >= 1 && c <= d - 1 && (r + c) % 2 == 0;
            const bool lr = (c == 0 || c == d) && r >= 1 && r <= d - 1 && (r + c) % 2 == 1;
            if (inner || tb || lr) cells.emplace_back(r, c);
        }
    return cells;
}

// Weight streams of the token kernel: the A fragments of each GEMM in the order the kernel
// consumes them. post: Wo (row tile, k-step), then per feed-forward chunk c the W1
// fragments of its CH hidden units (row tile, k-step) followed by the W2 fragments of its
// k-steps (row tile, k-step). qkv: per 32-feature output group og, per k-step, the two
// row tiles 2og and 2og+1.
void append_post_stream(std::vector<uint16_t>& out, const float* Wo, const float* W1, const float* W2, int D, int F,
                        int CH) {
    const int RT = D / 16, KS = D / 32, FKS = F / 32;
    std::vector<uint16_t> fo, f1, f2;
    append_frags(fo, Wo, D, D);
    append_frags(f1, W1, D, F);
    append_frags(f2, W2, F, D);
    auto frag = [&](const std::vector<uint16_t>& v, int ro, int ks, int nks) {
        out.insert(out.end(), v.begin() + ((size_t)ro * nks + ks) * 512, v.begin() + ((size_t)ro * nks + ks + 1) * 512);
    };
    for (int rt = 0; rt < RT; ++rt)
        for (int ks = 0; ks < KS; ++ks) frag(fo, rt, ks, KS);
    for (int c = 0; c < F / CH; ++c) {
        for (int rh = 0; rh < CH / 16; ++rh)
            for (int ks = 0; ks < KS; ++ks) frag(f1, c * (CH / 16) + rh, ks, KS);
        for (int rt = 0; rt < RT; ++rt)
            for (int kh = 0; kh < CH / 32; ++kh) frag(f2, rt, c * (CH / 32) + kh, FKS);
    }
}

void append_qkv_stream(std::vector<uint16_t>& out, const float* Wqkv, int D) {
    const int KS = D / 32;
    std::vector<uint16_t> f;
    append_frags(f, Wqkv, D, 3 * D);
    for (int og = 0; og < 3 * KS; ++og)
        for (int ks = 0; ks < KS; ++ks)
            for (int half = 0; half < 2; ++half) {
                const size_t fr = (size_t)(2 * og + half) * KS + ks;
                out.insert(out.end(), f.begin() + fr * 512, f.begin() + (fr + 1) * 512);
            }
}

// ---- MXFP8 weight streams (PWD_DTYPE_MXFP8; OCP Microscaling v1.0: E4M3 elements, one E8M0
// scale per block of 32 input features)

// Block of input feature f: each 128-feature slice splits into four blocks of 32, the runs of 8
// features of a 64-feature half alternating between two of them -- the blocks whose scales the
// token kernel's matrix-core operands take from lane groups 0..3 (see tok.hip).
int mx_block(int f) { return 4 * (f / 128) + 2 * ((f / 64) % 2) + (f / 8) % 2; }

// Shared exponent of a block with largest magnitude amax: floor(log2 amax) - 8 (8: the exponent
// of E4M3's largest power of two), within E8M0's [-127, 127]; -127 for amax = 0.
int mx_exponent(double amax) {
    if (!(amax > 0.0)) return -127;
    int e;
    std::frexp(amax, &e);   // amax = m 2^e, m in [0.5, 1): floor(log2 amax) = e - 1
    return std::min(127, std::max(-127, e - 1 - 8));
}

// E4M3 code of v: nearest value, ties to even mantissa; magnitudes from 448 (the largest finite
// value) up clamp to 448. Codes are monotone in the magnitude, subnormals (2^-9 steps below
// 2^-6) included.
uint8_t e4m3_code(double v) {
    const uint8_t sign = std::signbit(v) ? 0x80 : 0x00;
    const double a = std::fabs(v);
    if (!(a < 448.0)) return sign | 0x7e;
    if (a < std::ldexp(1.0, -6)) return sign | (uint8_t)std::nearbyint(std::ldexp(a, 9));   // 8 -> 2^-6
    int e;
    std::frexp(a, &e);
    int E = e - 1;                                              // a in [2^E, 2^(E+1)), E in [-6, 8]
    int q = (int)std::nearbyint((std::ldexp(a, -E) - 1.0) * 8.0);   // 3 mantissa bits
    if (q == 8) {
        q = 0;
        ++E;
    }
    return sign | (uint8_t)(((E + 7) << 3) | q);
}

// Exponents [O][K/32] of W [K][O] (y = x W), one per output feature and input block.
std::vector<int> mx_exponents(const float* W, int K, int O) {
    std::vector<double> amax((size_t)O * (K / 32), 0.0);
    for (int k = 0; k < K; ++k)
        for (int o = 0; o < O; ++o) {
            double& m = amax[(size_t)o * (K / 32) + mx_block(k)];
            m = std::max(m, std::fabs((double)W[(size_t)k * O + o]));
        }
    std::vector<int> ex(amax.size());
    for (size_t i = 0; i < amax.size(); ++i) ex[i] = mx_exponent(amax[i]);
    return ex;
}

// The 8-bit A fragment (row tile ro, 128-deep k-step ks8) of W^T: 2 KB at `frag`, half h of lane
// l at frag + 1024 h + 16 l; lane (m = l % 16, g = l / 16) byte e holds input feature
// 128 ks8 + 16 (e / 4) + 4 g + e % 4 of output feature 16 ro + m, divided by its block's scale.
// scale[16 l]: the E8M0 byte (exponent + 127) of output 16 ro + m, block 4 ks8 + g -- the
// block lane group g stands for.
void mx_fragment(const float* W, int K, int O, const std::vector<int>& ex, int ro, int ks8, uint8_t* frag,
                 uint8_t* scale) {
    for (int l = 0; l < 64; ++l) {
        const int m = l & 15, g = l >> 4, o = 16 * ro + m;
        for (int e = 0; e < 32; ++e) {
            const int k = 128 * ks8 + 16 * (e / 4) + 4 * g + e % 4;
            const double v = std::ldexp((double)W[(size_t)k * O + o], -ex[(size_t)o * (K / 32) + mx_block(k)]);
            frag[1024 * (e / 16) + 16 * l + e % 16] = e4m3_code(v);
        }
        scale[16 * l] = (uint8_t)(ex[(size_t)o * (K / 32) + 4 * ks8 + g] + 127);
    }
}

// MXFP8 Q/K/V stream of one layer (Wqkv [D][3D]): chunks of 32 KB, each holding `per_chunk`
// 8-bit fragments (output group og of 32 features, k-step ks8, row tile 2 og + hh), then, in
// 1 KB slot `scale_slot`, byte j of each lane's 16 the scale of fragment j; unused bytes zero.
void append_qkv_stream_mx(std::vector<uint16_t>& out, const float* Wqkv, int D, int per_chunk, int scale_slot) {
    const int KS8 = D / 128, O = 3 * D, opc = per_chunk / (2 * KS8), nchunks = (O / 32) / opc;
    const std::vector<int> ex = mx_exponents(Wqkv, D, O);
    for (int qc = 0; qc < nchunks; ++qc) {
        std::vector<uint8_t> chunk(32 * 1024, 0);
        for (int j = 0; j < per_chunk; ++j) {
            const int hh = j & 1, ks8 = (j >> 1) % KS8, o2 = (j >> 1) / KS8;
            mx_fragment(Wqkv, D, O, ex, 2 * (qc * opc + o2) + hh, ks8, chunk.data() + 2048 * j,
                        chunk.data() + 1024 * scale_slot + j);
        }
        const size_t at = out.size();
        out.resize(at + chunk.size() / 2);
        std::memcpy(out.data() + at, chunk.data(), chunk.size());
    }
}

// MXFP8 post stream of one layer: the out-projection's bf16 fragments as in append_post_stream,
// then per feed-forward chunk of CH hidden units a 32 KB chunk: the 8-bit W1 fragments (hidden
// row tile, k-step), the bf16 W2 fragments (row tile, hidden k-step) right after them, and the
// W1 scales in slot `scale_slot`.
// Returns false if a chunk's data would reach the scale slot.
bool append_post_stream_mx(std::vector<uint16_t>& out, const float* Wo, const float* W1, const float* W2, int D, int F,
                           int CH, int scale_slot) {
    const int RT = D / 16, KS = D / 32, FKS = F / 32, KS8 = D / 128, nw1 = (CH / 16) * KS8;
    std::vector<uint16_t> fo, f2;
    append_frags(fo, Wo, D, D);
    append_frags(f2, W2, F, D);
    for (int rt = 0; rt < RT; ++rt)
        for (int ks = 0; ks < KS; ++ks)
            out.insert(out.end(), fo.begin() + ((size_t)rt * KS + ks) * 512, fo.begin() + ((size_t)rt * KS + ks + 1) * 512);
    const std::vector<int> ex = mx_exponents(W1, D, F);
    for (int c = 0; c < F / CH; ++c) {
        std::vector<uint8_t> chunk(32 * 1024, 0);
        for (int j = 0; j < nw1; ++j)
            mx_fragment(W1, D, F, ex, c * (CH / 16) + j / KS8, j % KS8, chunk.data() + 2048 * j,
                        chunk.data() + 1024 * scale_slot + j);
        int slot = 2 * nw1;
        for (int rt = 0; rt < RT; ++rt)
            for (int kh = 0; kh < CH / 32; ++kh, ++slot) {
                const size_t fr = (size_t)rt * FKS + c * (CH / 32) + kh;
                std::memcpy(chunk.data() + 1024 * slot, f2.data() + fr * 512, 1024);
            }
        if (slot > scale_slot) return false;
        const size_t at = out.size();
        out.resize(at + chunk.size() / 2);
        std::memcpy(out.data() + at, chunk.data(), chunk.size());
    }
    return true;
}

// The resident kernel's stream of one layer (d_model D, feed-forward width F): per 32-feature
// group og, the Q, K and V fragments of the group (part, k-step, row tile 2 og + hh), then the
// out-projection's fragments at k-step og (row tile); per feed-forward chunk of 64 hidden units,
// W1 (k-step, hidden row tile) and W2 (hidden k-step, output row tile).
void append_resident_stream(std::vector<uint16_t>& out, const float* Wq, const float* Wk, const float* Wv,
                            const float* Wo, const float* W1, const float* W2, int D, int F) {
    const int RT = D / 16, KS = D / 32, FKS = F / 32, CH = 64;
    std::vector<uint16_t> fq, fk, fv, fo, f1, f2;
    append_frags(fq, Wq, D, D);
    append_frags(fk, Wk, D, D);
    append_frags(fv, Wv, D, D);
    append_frags(fo, Wo, D, D);
    append_frags(f1, W1, D, F);
    append_frags(f2, W2, F, D);
    auto frag = [&](const std::vector<uint16_t>& v, int ro, int ks, int nks) {
        out.insert(out.end(), v.begin() + ((size_t)ro * nks + ks) * 512, v.begin() + ((size_t)ro * nks + ks + 1) * 512);
    };
    for (int og = 0; og < KS; ++og) {
        for (const auto* f : {&fq, &fk, &fv})
            for (int ks = 0; ks < KS; ++ks)
                for (int hh = 0; hh < 2; ++hh) frag(*f, 2 * og + hh, ks, KS);
        for (int rt = 0; rt < RT; ++rt) frag(fo, rt, og, KS);
    }
    for (int c = 0; c < F / CH; ++c) {
        for (int ks = 0; ks < KS; ++ks)
            for (int rh = 0; rh < CH / 16; ++rh) frag(f1, c * (CH / 16) + rh, ks, KS);
        for (int kh = 0; kh < CH / 32; ++kh)
            for (int rt = 0; rt < RT; ++rt) frag(f2, rt, c * (CH / 32) + kh, FKS);
    }
}

size_t layer_floats(int D, int F) { return (size_t)4 * D * D + 2 * (size_t)D * F + F + 9 * (size_t)D; }

bool has_conv(const pwd_model_dims* m) {
    return m->conv_dilation[0] != 0 || m->conv_dilation[1] != 0 || m->conv_dilation[2] != 0;
}
// blob floats of the embedder's Conv1d block and of the dilated convolutions (after beta)
size_t res_floats(const pwd_model_dims* m) {
    return m->embedder == PWD_EMBED_RESNET ? 6 * (size_t)m->d_model * m->d_model + 2 * (size_t)m->d_model : 0;
}
size_t conv_floats(const pwd_model_dims* m) {
    const size_t D = m->d_model;
    return has_conv(m) ? (size_t)m->n_layers * (27 * D * D + 3 * D) : 0;
}

// The embedder's residual block (model table: 2 x Conv1d(D, D) after Linear(1 -> D); the
// syndrome-convolution section puts it on the flattened (d+1)^2 array ahead of PE) as a
// lookup. Its input at cell q is E(q) = e_q w_e + b_e, one event bit lifted to D features,
// and zero outside the array (padding 1). Two kernel-3 layers make the output at cell c,
//   R(c) = b2 + sum_{k=-1..1} [c+k in range] h(c+k) Wr2[k+1],
//   h(p) = ReLU(b1 + sum_{k=-1..1} [p+k in range] E(p+k) Wr1[k+1]),
// a function of the event bits at cells c-2 .. c+2 and of which of those cells exist; the
// latter is one of five position classes (c = 0, c = 1, interior, c = L-2, c = L-1 with
// L = (d+1)^2 >= 16). tab[class * 32 + bits] = R in double precision, rounded once.
// nb[token] = the stabilizers at cells c-2 .. c+2 (-1: empty cell or outside), the class.
void emb_tables(const std::vector<std::pair<int, int>>& cells, const std::vector<int>& cell_stab, int d,
                int D, const float* w_e, const float* b_e, const float* res, std::vector<int>& nb,
                std::vector<float>& tab) {
    const int L = (d + 1) * (d + 1);
    const float *W1 = res, *b1 = W1 + 3 * (size_t)D * D, *W2 = b1 + D, *b2 = W2 + 3 * (size_t)D * D;
    auto cls_of = [&](int c) { return c == 0 ? 0 : c == 1 ? 1 : c == L - 2 ? 3 : c == L - 1 ? 4 : 2; };
    nb.assign(cells.size() * 8, 0);
    for (size_t s = 0; s < cells.size(); ++s) {
        const int c = cells[s].first * (d + 1) + cells[s].second;
        for (int j = 0; j < 5; ++j) {
            const int q = c + j - 2;
            nb[s * 8 + j] = q >= 0 && q < L ? cell_stab[q] : -1;
        }
        nb[s * 8 + 5] = cls_of(c);
    }
    const int rep_cell[5] = {0, 1, 2, L - 2, L - 1};
    tab.assign((size_t)5 * 32 * D, 0.f);
    std::vector<double> E(5 * (size_t)D), h(3 * (size_t)D), R(D);
    for (int cls = 0; cls < 5; ++cls) {
        const int c = rep_cell[cls];
        auto in_range = [&](int off) { return c + off >= 0 && c + off < L; };
        for (int pat = 0; pat < 32; ++pat) {
            for (int j = 0; j < 5; ++j)   // E at offsets -2 .. 2
                for (int f = 0; f < D; ++f)
                    E[j * D + f] = in_range(j - 2) ? ((pat >> j) & 1) * (double)w_e[f] + b_e[f] : 0.0;
            for (int pp = 0; pp < 3; ++pp) {   // h at offsets -1 .. 1
                double* hp = &h[pp * D];
                for (int o = 0; o < D; ++o) hp[o] = b1[o];
                for (int k = 0; k < 3; ++k) {
                    const int off = pp - 1 + k - 1;   // input offset
                    if (!in_range(off)) continue;
                    const double* x = &E[(off + 2) * D];
                    const float* Wk = W1 + (size_t)k * D * D;
                    for (int i = 0; i < D; ++i)
                        for (int o = 0; o < D; ++o) hp[o] += x[i] * Wk[(size_t)i * D + o];
                }
                for (int o = 0; o < D; ++o) hp[o] = in_range(pp - 1) ? std::max(hp[o], 0.0) : 0.0;
            }
            for (int o = 0; o < D; ++o) R[o] = b2[o];
            for (int k = 0; k < 3; ++k) {
                if (!in_range(k - 1)) continue;
                const double* x = &h[k * D];
                const float* Wk = W2 + (size_t)k * D * D;
                for (int i = 0; i < D; ++i)
                    for (int o = 0; o < D; ++o) R[o] += x[i] * Wk[(size_t)i * D + o];
            }
            for (int o = 0; o < D; ++o) tab[((size_t)cls * 32 + pat) * D + o] = (float)R[o];
        }
    }
}

// Scratch of decode_windows_noalloc: the activations (X, Q/K/V, Y and the convolutions' G) of a
// batch, in device memory the library reserves when it is loaded, so that the entry point needs
// no allocation. Each GPU holds its own copy; its address is looked up once per device.
static __device__ __align__(256) unsigned char scratch[PWD_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

// The device address of `scratch` on `device` (which must be current); looked up on first use.
int scratch_on(int device, void** out) {
    if (device < 0 || device >= 64) return fail(PWD_EHIP, "device %d out of range", device);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(PWD_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return PWD_OK;
}

}  // namespace

struct pwd_decoder {
    int device = 0;
    int d = 0, W = 0, max_windows = 0, N = 0, Npad = 0, nbw = 0, words = 0, b_left = 0;
    int ntok = 0;                  // tokens per window (N stabilizers, or (d+1)^2 grid cells)
    const int* tok_stab = nullptr; // grid token set: stabilizer of each token or -1
    int D = 0, L = 0, H = 0, F = 0, dh = 0, dtype = 0;
    float kappa = 0.f, eps = 0.f;
    int64_t n_tb_alloc = 0;
    // device memory
    void* weights = nullptr;       // one allocation for every parameter table
    float* X = nullptr;
    uint16_t* QKV = nullptr;
    uint16_t* Y = nullptr;
    uint16_t* G[2] = {nullptr, nullptr};   // dilated convolutions: bf16 token-major unit inputs
    int dil[3] = {0, 0, 0};        // their dilations (0: none)
    size_t conv_off = 0;           // fp32 path: float offset of their tensors in the blob
    int* err = nullptr;
    void* static_scratch = nullptr;   // device address of `scratch` on this device
    // decode_stream scratch: the windows cut from a stream and their results
    uint32_t* stream_meas = nullptr;   // [max_windows][W + 1][words]
    uint8_t* stream_types = nullptr;   // [max_windows]
    float* stream_logits = nullptr;    // [max_windows]
    uint8_t* stream_bits = nullptr;    // [max_windows]
    // views into `weights`
    struct Layer {
        const uint16_t *post, *qkv;
        const float *post_vecs, *bqkv;   // [b_o g1 be1 b2 g2 be2 | b1] (6 D + F) and [b_q b_k | b_v x rep]
        const uint16_t* conv[3] = {nullptr, nullptr, nullptr};   // dilated units: weight streams
        const float* conv_b[3] = {nullptr, nullptr, nullptr};    // and biases
    };
    std::vector<Layer> layers;
    const float* S0 = nullptr;
    const float* we = nullptr;
    const uint16_t* Wc = nullptr;
    const float* bc = nullptr;
    const float* wo = nullptr;
    const uint16_t* zero = nullptr;   // dilated convolutions: D zero values (off-grid neighbours)
    const int* cell_token = nullptr;
    const int* emb_nb = nullptr;   // embedder residual block (PWD_EMBED_RESNET): see emb_tables
    const float* emb_tab = nullptr;
    const float* f32w = nullptr;   // fp32 path: the blob tensors as given
    // the state-resident schedule (PWD_SCHEDULE_RESIDENT), when the configuration allows it
    bool resident_ok = false;
    int schedule = PWD_SCHEDULE_AUTO;
    int mlp_ratio = 4;
    const uint16_t* res_stream = nullptr;
    const float* res_vecs = nullptr;
    float bo_out = 0.f, beta[3] = {0.f, 0.f, 0.f};
    // per-stage timing (decoder_profile)
    bool profiling = false;
    struct Mark { hipEvent_t begin, end; int stage; };
    std::vector<Mark> marks;       // recorded, not yet read
    std::vector<hipEvent_t> spare; // released events for reuse
};

namespace {

hipEvent_t take_event(pwd_decoder* dec) {
    if (!dec->spare.empty()) {
        hipEvent_t e = dec->spare.back();
        dec->spare.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Launches `launch` on stream s; with profiling on, brackets it with an event pair.
template <class Fn>
hipError_t timed(pwd_decoder* dec, int stage, hipStream_t s, Fn launch) {
    if (!dec->profiling) return launch();
    hipEvent_t b = take_event(dec), e = take_event(dec);
    if (!b || !e) return hipErrorOutOfMemory;
    hipError_t err = hipEventRecord(b, s);
    if (err == hipSuccess) err = launch();
    if (err == hipSuccess) err = hipEventRecord(e, s);
    if (err != hipSuccess) return err;
    dec->marks.push_back({b, e, stage});
    return hipSuccess;
}

}  // namespace

extern "C" {

const char* decoder_last_error(void) { return g_last_error.c_str(); }

size_t decoder_blob_floats(const pwd_geometry* geom, const pwd_model_dims* dims) {
    if (!geom || !dims) return 0;
    const int D = dims->d_model, F = dims->mlp_ratio * dims->d_model, d = geom->distance;
    return 2 * (size_t)D + (size_t)dims->n_layers * layer_floats(D, F) + 4 * (size_t)D * D + D +
           (size_t)d * D + 1 + 3 + res_floats(dims) + conv_floats(dims);
}

int decoder_validate_config(const pwd_geometry* g, const pwd_model_dims* m) {
    if (!g || !m) return fail(PWD_EINVAL, "null geometry or dimensions");
    const int d = g->distance;
    // any odd distance whose attention tile (bf16) or window (fp32) fits on chip, checked below
    if (d < 3 || d > 63 || d % 2 == 0) return fail(PWD_EUNSUPPORTED, "distance %d: need odd 3..63", d);
    if (g->window_rounds < d || g->window_rounds > 3 * d)
        return fail(PWD_EUNSUPPORTED, "window_rounds %d: need %d..%d", g->window_rounds, d, 3 * d);
    if (g->max_windows < 1 || g->max_windows > (1 << 24))
        return fail(PWD_EUNSUPPORTED, "max_windows %d: need 1..2^24", g->max_windows);
    if (m->mlp_ratio != 4 && m->mlp_ratio != 5)
        return fail(PWD_EUNSUPPORTED, "mlp_ratio %d: need 4 or 5", m->mlp_ratio);
    if (m->n_layers < 1 || m->n_layers > 8) return fail(PWD_EUNSUPPORTED, "n_layers %d: need 1..8", m->n_layers);
    if (m->n_heads < 1 || m->d_model % m->n_heads != 0)
        return fail(PWD_EUNSUPPORTED, "d_model %d not divisible by n_heads %d", m->d_model, m->n_heads);
    const int dh = m->d_model / m->n_heads;
    if (m->token_set != PWD_TOKENS_STABILIZERS && m->token_set != PWD_TOKENS_GRID)
        return fail(PWD_EUNSUPPORTED, "token_set %d: need 0 (stabilizers) or 1 (grid)", m->token_set);
    if (m->embedder != PWD_EMBED_LINEAR && m->embedder != PWD_EMBED_RESNET)
        return fail(PWD_EUNSUPPORTED, "embedder %d: need 0 (linear) or 1 (linear + residual Conv1d)", m->embedder);
    if (has_conv(m)) {
        for (int j = 0; j < 3; ++j)
            if (m->conv_dilation[j] < 1 || m->conv_dilation[j] > d)
                return fail(PWD_EUNSUPPORTED, "conv_dilation[%d] = %d: need 1..%d (or all three 0)", j,
                            m->conv_dilation[j], d);
        if (m->token_set != PWD_TOKENS_GRID)
            return fail(PWD_EUNSUPPORTED, "dilated convolutions need the grid token set (every cell a token)");
        if (m->dtype == PWD_DTYPE_MXFP8)
            return fail(PWD_EUNSUPPORTED, "MXFP8 networks without the dilated convolutions only");
    }
    const int N = m->token_set == PWD_TOKENS_GRID ? (d + 1) * (d + 1) : d * d - 1;   // tokens
    if (m->dtype == PWD_DTYPE_BF16 || m->dtype == PWD_DTYPE_MXFP8) {
        if (m->d_model != 128 && m->d_model != 256)
            return fail(PWD_EUNSUPPORTED, "bf16 d_model %d: need 128 or 256", m->d_model);
        if (dh != 16 && dh != 32 && dh != 64)
            return fail(PWD_EUNSUPPORTED, "bf16 head size %d: need 16, 32 or 64", dh);
        const size_t smem = attn_smem_bytes(dh, (N + 15) / 16 * 16, (N + 15) / 16);
        if (smem > 160 * 1024) return fail(PWD_EUNSUPPORTED, "attention tile needs %zu bytes of LDS", smem);
    } else if (m->dtype == PWD_DTYPE_F32) {
        if (m->d_model != 16 && m->d_model != 32 && m->d_model != 64)
            return fail(PWD_EUNSUPPORTED, "fp32 d_model %d: need 16, 32 or 64", m->d_model);
        if (dh != 4 && dh != 8 && dh != 16 && dh != 32 && dh != 64)
            return fail(PWD_EUNSUPPORTED, "fp32 head size %d: need 4, 8, 16, 32 or 64", dh);
        const size_t smem = f32_window_smem_bytes(N, m->d_model, m->n_heads, m->mlp_ratio * m->d_model);
        if (smem > 64 * 1024)
            return fail(PWD_EUNSUPPORTED, "fp32 window of %d tokens needs %zu bytes of LDS (max 65536)", N, smem);
    } else {
        return fail(PWD_EUNSUPPORTED, "dtype %d: need 0 (fp32), 1 (bf16) or 2 (MXFP8)", m->dtype);
    }
    return PWD_OK;
}

int decoder_create(const pwd_geometry* geom, const pwd_model_dims* dims, const void* blob,
                   size_t blob_bytes, pwd_decoder** out) {
    if (!out || !blob) return fail(PWD_EINVAL, "null blob or output handle");
    int rc = decoder_validate_config(geom, dims);
    if (rc != PWD_OK) return rc;
    const size_t nf = decoder_blob_floats(geom, dims);
    if (blob_bytes != PWD_BLOB_HEADER_WORDS * 4 + nf * 4)
        return fail(PWD_EBLOB, "blob has %zu bytes, expected %zu", blob_bytes, PWD_BLOB_HEADER_WORDS * 4 + nf * 4);
    uint32_t hdr[PWD_BLOB_HEADER_WORDS];
    std::memcpy(hdr, blob, sizeof hdr);
    const int d = geom->distance, D = dims->d_model, L = dims->n_layers, H = dims->n_heads;
    const int F = dims->mlp_ratio * D;
    if (hdr[0] != PWD_BLOB_MAGIC) return fail(PWD_EBLOB, "bad blob magic 0x%08x", hdr[0]);
    if (hdr[1] != PWD_BLOB_VERSION) return fail(PWD_EBLOB, "blob version %u, expected %d", hdr[1], PWD_BLOB_VERSION);
    const int expect[7] = {d, geom->window_rounds, D, L, H, F, dims->dtype};
    for (int i = 0; i < 7; ++i)
        if ((int)hdr[2 + i] != expect[i])
            return fail(PWD_EBLOB, "blob header word %d is %d, expected %d", 2 + i, (int)hdr[2 + i], expect[i]);
    if ((int)hdr[11] != dims->token_set)
        return fail(PWD_EBLOB, "blob header word 11 (token set) is %d, expected %d", (int)hdr[11], dims->token_set);
    if ((int)hdr[12] != dims->embedder)
        return fail(PWD_EBLOB, "blob header word 12 (embedder) is %d, expected %d", (int)hdr[12], dims->embedder);
    const uint32_t dil_word = (uint32_t)dims->conv_dilation[0] | ((uint32_t)dims->conv_dilation[1] << 8) |
                              ((uint32_t)dims->conv_dilation[2] << 16);
    if (hdr[13] != dil_word)
        return fail(PWD_EBLOB, "blob header word 13 (dilations) is 0x%x, expected 0x%x", hdr[13], dil_word);
    float kappa, eps;
    std::memcpy(&kappa, &hdr[9], 4);
    std::memcpy(&eps, &hdr[10], 4);
    if (!(eps > 0.f) || !std::isfinite(kappa)) return fail(PWD_EBLOB, "blob kappa/eps invalid");
    const float* wf = reinterpret_cast<const float*>(static_cast<const char*>(blob) + PWD_BLOB_HEADER_WORDS * 4);
    std::vector<float> w(wf, wf + nf);   // aligned copy

    int device = 0;
    HIP_OK(hipGetDevice(&device));
    void* static_scratch = nullptr;   // decode_windows_noalloc's scratch on this device
    rc = scratch_on(device, &static_scratch);
    if (rc != PWD_OK) return rc;
    pwd_decoder* dec = new (std::nothrow) pwd_decoder();
    if (!dec) return fail(PWD_ENOMEM, "host allocation failed");
    dec->device = device;
    dec->static_scratch = static_scratch;
    dec->d = d;
    dec->W = geom->window_rounds;
    dec->max_windows = geom->max_windows;
    const bool grid = dims->token_set == PWD_TOKENS_GRID;
    dec->N = d * d - 1;
    dec->ntok = grid ? (d + 1) * (d + 1) : dec->N;
    dec->Npad = (dec->ntok + 15) / 16 * 16;
    dec->nbw = dec->Npad / 16;
    dec->words = (dec->N + 31) / 32;
    dec->b_left = (dec->W - d) / 2;
    dec->D = D; dec->L = L; dec->H = H; dec->F = F; dec->dh = D / H; dec->dtype = dims->dtype;
    dec->kappa = kappa; dec->eps = eps;
    for (int j = 0; j < 3; ++j) dec->dil[j] = dims->conv_dilation[j];

    // geometry tables: the cell of each token (grid: every cell, row-major), each cell's
    // token (-1: none), and for the grid token set each token's stabilizer (-1: none)
    const auto stab_cells = stabilizer_cells(d);
    std::vector<std::pair<int, int>> cells = stab_cells;
    std::vector<int> tok_stab;
    if (grid) {
        cells.clear();
        tok_stab.assign((size_t)(d + 1) * (d + 1), -1);
        for (int r = 0; r <= d; ++r)
            for (int c = 0; c <= d; ++c) cells.push_back({r, c});
        for (size_t s = 0; s < stab_cells.size(); ++s)
            tok_stab[stab_cells[s].first * (d + 1) + stab_cells[s].second] = (int)s;
    }
    std::vector<int> cell_token((size_t)(d + 1) * (d + 1), -1);
    for (size_t s = 0; s < cells.size(); ++s) cell_token[cells[s].first * (d + 1) + cells[s].second] = (int)s;

    // the parameter tables, laid out in one host image, then one upload
    std::vector<unsigned char> img;
    auto align = [&]() { img.resize((img.size() + 255) & ~(size_t)255); };
    auto put = [&](const void* src, size_t bytes) {
        align();
        const size_t off = img.size();
        img.resize(off + bytes);
        std::memcpy(img.data() + off, src, bytes);
        return off;
    };

    // S0 = b_e + PE[pos(s)] (App. A.1.4 sinusoids over the flattened lattice index), double
    // precision on the host, rounded to fp32.
    const float* b_e = w.data() + D;
    std::vector<double> pe_row(D);
    auto pe_of = [&](int pos) {
        for (int i = 0; i < D / 2; ++i) {
            const double ang = pos / std::pow(10000.0, 2.0 * i / D);
            pe_row[2 * i] = std::sin(ang);
            pe_row[2 * i + 1] = std::cos(ang);
        }
    };
    const size_t off_cell = put(cell_token.data(), cell_token.size() * sizeof(int));
    const size_t off_tok_stab = grid ? put(tok_stab.data(), tok_stab.size() * sizeof(int)) : 0;
    size_t off_emb_nb = 0, off_emb_tab = 0;
    if (dims->embedder == PWD_EMBED_RESNET) {
        std::vector<int> cell_stab((size_t)(d + 1) * (d + 1), -1);
        for (size_t s = 0; s < stab_cells.size(); ++s)
            cell_stab[stab_cells[s].first * (d + 1) + stab_cells[s].second] = (int)s;
        std::vector<int> nb;
        std::vector<float> tab;
        const float* res = w.data() + nf - conv_floats(dims) - res_floats(dims);   // after beta
        emb_tables(cells, cell_stab, d, D, w.data(), w.data() + D, res, nb, tab);
        off_emb_nb = put(nb.data(), nb.size() * sizeof(int));
        off_emb_tab = put(tab.data(), tab.size() * sizeof(float));
    }

    struct LayerOff { size_t post, qkv, post_vecs, bqkv, conv[3], conv_b[3]; };
    std::vector<LayerOff> loff(L);
    size_t off_S0 = 0, off_we = 0, off_Wc = 0, off_bc = 0, off_wo = 0, off_f32 = 0, off_zero = 0;
    size_t off_res_stream = 0, off_res_vecs = 0;
    const bool resident_ok = dims->dtype == PWD_DTYPE_BF16 && !has_conv(dims) && dims->embedder == PWD_EMBED_LINEAR &&
                             resident_supported(D, (dec->ntok + 15) / 16, L, dims->mlp_ratio, D / H);
    dec->resident_ok = resident_ok;
    dec->mlp_ratio = dims->mlp_ratio;
    const size_t lf = layer_floats(D, F);
    const float* tail = w.data() + 2 * D + (size_t)L * lf;   // Wc, bc, w_o, b_o, beta
    const bool mx = dims->dtype == PWD_DTYPE_MXFP8;
    if (dims->dtype != PWD_DTYPE_F32) {
        const int RT = D / 16;
        std::vector<float> s0((size_t)dec->nbw * RT * 64 * 4, 0.f);
        for (int s = 0; s < dec->ntok; ++s) {
            pe_of(cells[s].first * (d + 1) + cells[s].second);
            const int blk = s / 16, cl = s % 16;
            for (int f = 0; f < D; ++f) {
                const int rt = f / 16, g = (f % 16) / 4, i = f % 4;
                s0[(((size_t)blk * RT + rt) * 64 + g * 16 + cl) * 4 + i] = (float)((double)b_e[f] + pe_row[f]);
            }
        }
        off_S0 = put(s0.data(), s0.size() * 4);
        off_we = put(w.data(), (size_t)D * 4);
        for (int l = 0; l < L; ++l) {
            const float* p = w.data() + 2 * D + (size_t)l * lf;
            const float *Wq = p, *bq = Wq + D * D, *Wk = bq + D, *bk = Wk + D * D, *Wv = bk + D, *bv = Wv + D * D;
            const float *Wo = bv + D, *bo = Wo + D * D, *g1 = bo + D, *be1 = g1 + D, *W1 = be1 + D;
            const float *b1 = W1 + (size_t)D * F, *W2 = b1 + F, *b2 = W2 + (size_t)F * D, *g2 = b2 + D, *be2 = g2 + D;
            const int rep = tok_bv_rep(D, F);
            std::vector<float> wqkv((size_t)D * 3 * D), bqkv((size_t)(2 + rep) * D);
            for (int k = 0; k < D; ++k)
                for (int o = 0; o < D; ++o) {
                    wqkv[(size_t)k * 3 * D + o] = Wq[k * D + o];
                    wqkv[(size_t)k * 3 * D + D + o] = Wk[k * D + o];
                    wqkv[(size_t)k * 3 * D + 2 * D + o] = Wv[k * D + o];
                }
            for (int o = 0; o < D; ++o) {
                bqkv[o] = bq[o];
                bqkv[D + o] = bk[o];
                for (int r = 0; r < rep; ++r) bqkv[2 * D + rep * o + r] = bv[o];
            }
            std::vector<uint16_t> fr;
            if (mx) {
                if (!append_post_stream_mx(fr, Wo, W1, W2, D, F, tok_mlp_chunk(D), tok_mx_scale_slot())) {
                    delete dec;
                    return fail(PWD_EUNSUPPORTED, "MXFP8 feed-forward chunk layout does not fit");
                }
            } else {
                append_post_stream(fr, Wo, W1, W2, D, F, tok_mlp_chunk(D));
            }
            loff[l].post = put(fr.data(), fr.size() * 2);
            fr.clear();
            if (mx) append_qkv_stream_mx(fr, wqkv.data(), D, tok_mx_qkv_frags(), tok_mx_scale_slot());
            else append_qkv_stream(fr, wqkv.data(), D);
            loff[l].qkv = put(fr.data(), fr.size() * 2);
            std::vector<float> pv;   // the token kernel's LDS vector table order
            for (const float* v : {bo, g1, be1, b2, g2, be2}) pv.insert(pv.end(), v, v + D);
            pv.insert(pv.end(), b1, b1 + F);
            loff[l].post_vecs = put(pv.data(), pv.size() * 4);
            loff[l].bqkv = put(bqkv.data(), bqkv.size() * 4);
            if (has_conv(dims)) {
                // dilated unit j: 9 taps, each the A fragments of Wd[j][a][e]^T in
                // (row tile, k-step) order, the order the convolution kernel consumes them
                const float* cw = w.data() + nf - conv_floats(dims) + (size_t)l * (27 * (size_t)D * D + 3 * D);
                for (int j = 0; j < 3; ++j) {
                    fr.clear();
                    for (int tap = 0; tap < 9; ++tap) append_frags(fr, cw + ((size_t)j * 9 + tap) * D * D, D, D);
                    loff[l].conv[j] = put(fr.data(), fr.size() * 2);
                    loff[l].conv_b[j] = put(cw + 27 * (size_t)D * D + (size_t)j * D, (size_t)D * 4);
                }
            }
        }
        if (resident_ok) {
            std::vector<uint16_t> rs;
            std::vector<float> rv;
            for (int l = 0; l < L; ++l) {
                const float* p = w.data() + 2 * D + (size_t)l * lf;
                const float *Wq = p, *bq = Wq + D * D, *Wk = bq + D, *bk = Wk + D * D, *Wv = bk + D, *bv = Wv + D * D;
                const float *Wo = bv + D, *bo = Wo + D * D, *g1 = bo + D, *be1 = g1 + D, *W1 = be1 + D;
                const float *b1 = W1 + (size_t)D * F, *W2 = b1 + F, *b2 = W2 + (size_t)F * D, *g2 = b2 + D, *be2 = g2 + D;
                append_resident_stream(rs, Wq, Wk, Wv, Wo, W1, W2, D, F);
                for (const float* v : {bq, bk, bv, bo, g1, be1, b2, g2, be2}) rv.insert(rv.end(), v, v + D);
                rv.insert(rv.end(), b1, b1 + F);
            }
            off_res_stream = put(rs.data(), rs.size() * 2);
            off_res_vecs = put(rv.data(), rv.size() * 4);
        }
        {
            std::vector<uint16_t> fr;
            append_frags(fr, tail, 4 * D, D);   // Wc[2][2][D][D] read as [4D][D]
            off_Wc = put(fr.data(), fr.size() * 2);
        }
        off_bc = put(tail + 4 * (size_t)D * D, D * 4);
        if (has_conv(dims)) {
            const std::vector<uint16_t> zeros((size_t)D, 0);
            off_zero = put(zeros.data(), zeros.size() * 2);
        }
        off_wo = put(tail + 4 * (size_t)D * D + D, (size_t)d * D * 4);
    } else {
        std::vector<float> s0((size_t)dec->ntok * D);
        for (int s = 0; s < dec->ntok; ++s) {
            pe_of(cells[s].first * (d + 1) + cells[s].second);
            for (int f = 0; f < D; ++f) s0[(size_t)s * D + f] = (float)((double)b_e[f] + pe_row[f]);
        }
        off_S0 = put(s0.data(), s0.size() * 4);
        off_f32 = put(w.data(), nf * 4);
        dec->conv_off = nf - conv_floats(dims);
    }
    const float* bo_beta = tail + 4 * (size_t)D * D + D + (size_t)d * D;
    dec->bo_out = bo_beta[0];
    for (int i = 0; i < 3; ++i) dec->beta[i] = bo_beta[1 + i];

    auto cleanup_fail = [&](int code) {
        decoder_destroy(dec);
        return code;
    };
    hipError_t e = hipMalloc(&dec->weights, img.size());
    if (e != hipSuccess) return cleanup_fail(fail(PWD_ENOMEM, "hipMalloc(weights, %zu): %s", img.size(), hipGetErrorString(e)));
    e = hipMemcpy(dec->weights, img.data(), img.size(), hipMemcpyHostToDevice);
    if (e != hipSuccess) return cleanup_fail(fail(PWD_EHIP, "hipMemcpy(weights): %s", hipGetErrorString(e)));
    e = hipMalloc(&dec->err, sizeof(int));
    if (e == hipSuccess) e = hipMemset(dec->err, 0, sizeof(int));
    if (e != hipSuccess) return cleanup_fail(fail(PWD_ENOMEM, "error word: %s", hipGetErrorString(e)));

    const unsigned char* base = static_cast<const unsigned char*>(dec->weights);
    auto fptr = [&](size_t off) { return reinterpret_cast<const float*>(base + off); };
    auto hptr = [&](size_t off) { return reinterpret_cast<const uint16_t*>(base + off); };
    dec->cell_token = reinterpret_cast<const int*>(base + off_cell);
    if (grid) dec->tok_stab = reinterpret_cast<const int*>(base + off_tok_stab);
    if (dims->embedder == PWD_EMBED_RESNET) {
        dec->emb_nb = reinterpret_cast<const int*>(base + off_emb_nb);
        dec->emb_tab = fptr(off_emb_tab);
    }
    dec->S0 = fptr(off_S0);
    if (dims->dtype != PWD_DTYPE_F32) {
        dec->we = fptr(off_we);
        dec->Wc = hptr(off_Wc);
        dec->bc = fptr(off_bc);
        if (has_conv(dims)) dec->zero = hptr(off_zero);
        dec->wo = fptr(off_wo);
        if (resident_ok) {
            dec->res_stream = hptr(off_res_stream);
            dec->res_vecs = fptr(off_res_vecs);
        }
        for (int l = 0; l < L; ++l) {
            pwd_decoder::Layer ly;
            ly.post = hptr(loff[l].post); ly.qkv = hptr(loff[l].qkv);
            ly.post_vecs = fptr(loff[l].post_vecs);
            ly.bqkv = fptr(loff[l].bqkv);
            if (has_conv(dims))
                for (int j = 0; j < 3; ++j) {
                    ly.conv[j] = hptr(loff[l].conv[j]);
                    ly.conv_b[j] = fptr(loff[l].conv_b[j]);
                }
            dec->layers.push_back(ly);
        }
        const int64_t gran = tok_block_granule();
        dec->n_tb_alloc = ((int64_t)dec->max_windows * dec->nbw + gran - 1) / gran * gran;
        const size_t xb = (size_t)dec->n_tb_alloc * 16 * D * sizeof(float);
        const size_t qb = (size_t)dec->n_tb_alloc * 48 * D * sizeof(uint16_t);
        const size_t yb = (size_t)dec->n_tb_alloc * 16 * D * sizeof(uint16_t);
        if ((e = hipMalloc(&dec->X, xb)) != hipSuccess || (e = hipMalloc(&dec->QKV, qb)) != hipSuccess ||
            (e = hipMalloc(&dec->Y, yb)) != hipSuccess)
            return cleanup_fail(fail(PWD_ENOMEM, "scratch for %d windows (%zu bytes): %s", dec->max_windows,
                                     xb + qb + yb, hipGetErrorString(e)));
        // padding blocks are computed too; start them from finite values
        if ((e = hipMemset(dec->X, 0, xb)) != hipSuccess || (e = hipMemset(dec->QKV, 0, qb)) != hipSuccess ||
            (e = hipMemset(dec->Y, 0, yb)) != hipSuccess)
            return cleanup_fail(fail(PWD_EHIP, "scratch clear: %s", hipGetErrorString(e)));
        if (has_conv(dims))
            for (int i = 0; i < 2; ++i) {
                if ((e = hipMalloc(&dec->G[i], yb)) != hipSuccess)
                    return cleanup_fail(fail(PWD_ENOMEM, "convolution buffers (%zu bytes): %s", 2 * yb,
                                             hipGetErrorString(e)));
                if ((e = hipMemset(dec->G[i], 0, yb)) != hipSuccess)
                    return cleanup_fail(fail(PWD_EHIP, "scratch clear: %s", hipGetErrorString(e)));
            }
    } else {
        dec->f32w = fptr(off_f32);
    }
    {
        const size_t mw = (size_t)dec->max_windows;
        const size_t mb = mw * (dec->W + 1) * dec->words * sizeof(uint32_t);
        if ((e = hipMalloc(&dec->stream_meas, mb)) != hipSuccess || (e = hipMalloc(&dec->stream_types, mw)) != hipSuccess ||
            (e = hipMalloc(&dec->stream_logits, mw * sizeof(float))) != hipSuccess ||
            (e = hipMalloc(&dec->stream_bits, mw)) != hipSuccess)
            return cleanup_fail(fail(PWD_ENOMEM, "stream scratch for %d windows: %s", dec->max_windows, hipGetErrorString(e)));
    }
    *out = dec;
    return PWD_OK;
}

int decoder_destroy(pwd_decoder* dec) {
    if (!dec) return PWD_OK;
    DeviceGuard dg(dec->device);
    (void)hipFree(dec->weights);
    (void)hipFree(dec->X);
    (void)hipFree(dec->QKV);
    (void)hipFree(dec->Y);
    (void)hipFree(dec->G[0]);
    (void)hipFree(dec->G[1]);
    (void)hipFree(dec->err);
    (void)hipFree(dec->stream_meas);
    (void)hipFree(dec->stream_types);
    (void)hipFree(dec->stream_logits);
    (void)hipFree(dec->stream_bits);
    for (auto& m : dec->marks) {
        (void)hipEventDestroy(m.begin);
        (void)hipEventDestroy(m.end);
    }
    for (auto e : dec->spare) (void)hipEventDestroy(e);
    delete dec;
    return PWD_OK;
}

static SyndromeIn syndrome_in(const pwd_decoder* dec, const uint32_t* meas, const uint8_t* types, int64_t n) {
    SyndromeIn in;
    in.meas = meas;
    in.types = types;
    in.nwin = (int)n;
    in.W = dec->W;
    in.words = dec->words;
    in.d = dec->d;
    in.N = dec->N;
    in.b_left = dec->b_left;
    return in;
}

// The activation buffers of one decode: the handle's own (sized for max_windows) or carved out
// of the static scratch (decode_windows_noalloc).
struct Activations {
    float* X;
    uint16_t* QKV;
    uint16_t* Y;
    uint16_t* G[2];
};

static Activations handle_activations(const pwd_decoder* dec) {
    return Activations{dec->X, dec->QKV, dec->Y, {dec->G[0], dec->G[1]}};
}

// Bytes of X, Q/K/V, Y (and the two G buffers with dilated convolutions) for n_tb token blocks.
static size_t activation_bytes(const pwd_decoder* dec, int64_t n_tb, size_t* xb, size_t* qb, size_t* yb) {
    *xb = (size_t)n_tb * 16 * dec->D * sizeof(float);
    *qb = (size_t)n_tb * 48 * dec->D * sizeof(uint16_t);
    *yb = (size_t)n_tb * 16 * dec->D * sizeof(uint16_t);
    return *xb + *qb + *yb + (dec->dil[0] ? 2 * *yb : 0);
}

static int check_batch(const pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types, int64_t n,
                       const float* d_logits, const uint8_t* d_bits) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    if (n < 0) return fail(PWD_EINVAL, "negative n_windows");
    if (n > dec->max_windows) return fail(PWD_EBATCH, "n_windows %lld > max_windows %d", (long long)n, dec->max_windows);
    if (n > 0 && (!d_meas || !d_types || !d_logits || !d_bits)) return fail(PWD_EINVAL, "null buffer");
    return PWD_OK;
}

// decode_windows with `readouts` readouts after the last `readouts` rounds (1: the inference
// branch; distance: the recurrent branch), written to d_logits[win * readouts + k].
static int decode_impl(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types, int64_t n,
                       float* d_logits, uint8_t* d_bits, void* hip_stream, int readouts, const Activations& act) {
    const int rc0 = check_batch(dec, d_meas, d_types, n, d_logits, d_bits);
    if (rc0 != PWD_OK) return rc0;
    if (n == 0) return PWD_OK;
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    const SyndromeIn in = syndrome_in(dec, d_meas, d_types, n);

    if (dec->dtype == PWD_DTYPE_F32) {
        F32Params p;
        p.in = in;
        p.w = dec->f32w;
        p.S0 = dec->S0;
        p.ntok = dec->ntok;
        p.tok_stab = dec->tok_stab;
        p.emb_nb = dec->emb_nb;
        p.emb_tab = dec->emb_tab;
        p.conv_w = dec->dil[0] ? dec->f32w + dec->conv_off : nullptr;
        for (int j = 0; j < 3; ++j) p.dil[j] = dec->dil[j];
        p.cell_token = dec->cell_token;
        p.logits = d_logits;
        p.bits = d_bits;
        p.err = dec->err;
        p.D = dec->D; p.L = dec->L; p.H = dec->H; p.F = dec->F;
        p.readouts = readouts;
        p.kappa = dec->kappa; p.eps = dec->eps;
        HIP_OK(timed(dec, PWD_STAGE_FP32_WINDOW, s, [&] { return launch_f32_window(p, s); }));
        return PWD_OK;
    }

    const int64_t n_tb = n * dec->nbw;
    ReadoutParams rp;
    rp.X = act.X;
    rp.Xb = nullptr;
    rp.types = d_types;
    rp.err = dec->err;
    rp.Wc = dec->Wc;
    rp.bc = dec->bc;
    rp.wo = dec->wo;
    rp.bo = dec->bo_out;
    for (int i = 0; i < 3; ++i) rp.beta[i] = dec->beta[i];
    rp.cell_token = dec->cell_token;
    rp.nwin = (int)n;
    rp.d = dec->d;
    rp.D = dec->D;
    rp.nbw = dec->nbw;
    rp.stride = readouts;
    // readout of D_t into output slot k; `state` is null for the fp32 final state in X, else
    // the bf16 copy of D_t
    auto readout = [&](int k, const uint16_t* state) {
        rp.Xb = state;
        rp.logits = d_logits + k;
        rp.bits = d_bits + k;
        return timed(dec, PWD_STAGE_READOUT, s, [&] { return launch_readout(rp, s); });
    };

    if (readouts == 1 && dec->resident_ok && dec->schedule != PWD_SCHEDULE_LAYERS) {
        ResidentParams rs;
        rs.in = in;
        rs.ntok = dec->ntok;
        rs.tok_stab = dec->tok_stab;
        rs.nbw = dec->nbw;
        rs.L = dec->L;
        rs.kappa = dec->kappa;
        rs.eps = dec->eps;
        rs.qscale = (float)(1.4426950408889634 / std::sqrt((double)dec->dh));
        rs.stream = dec->res_stream;
        rs.vecs = dec->res_vecs;
        rs.S0 = dec->S0;
        rs.we = dec->we;
        rs.X = act.X;
        HIP_OK(timed(dec, PWD_STAGE_RESIDENT, s, [&] { return launch_resident(dec->mlp_ratio, dec->dh, rs, s); }));
        HIP_OK(readout(0, nullptr));
        return PWD_OK;
    }

    TokParams tp;
    std::memset(&tp, 0, sizeof tp);
    tp.in = in;
    tp.Npad = dec->Npad;
    tp.nbw = dec->nbw;
    tp.kappa = dec->kappa;
    tp.eps = dec->eps;
    tp.qscale = (float)(1.4426950408889634 / std::sqrt((double)dec->dh));
    tp.X = act.X;
    tp.QKV = act.QKV;
    tp.Y = act.Y;
    tp.S0 = dec->S0;
    tp.ntok = dec->ntok;
    tp.tok_stab = dec->tok_stab;
    tp.emb_nb = dec->emb_nb;
    tp.emb_tab = dec->emb_tab;
    const int RES = dec->emb_tab ? TOK_RESNET : 0;
    const int MXF = dec->dtype == PWD_DTYPE_MXFP8 ? TOK_MX : 0;   // MXFP8 Q/K/V and W1
    tp.we = dec->we;
    auto set_post = [&](int l) {
        const auto& ly = dec->layers[l];
        tp.post_stream = ly.post;
        tp.post_vecs = ly.post_vecs;
    };
    auto set_qkv = [&](int l) {
        tp.qkv_stream = dec->layers[l].qkv;
        tp.bqkv = dec->layers[l].bqkv;
    };
    AttnParams ap;
    ap.QKV = act.QKV;
    ap.Y = act.Y;
    ap.N = dec->ntok;
    ap.Npad = dec->Npad;
    ap.nbw = dec->nbw;
    ap.H = dec->H;

    // POST of layer l followed by `flags` (QKV, EMBED, RESNET). With the dilated convolutions:
    // out-projection + LN1 (writing the first unit's input G), the three residual units
    // (G ping-pongs between two buffers; X is updated in place), then feed-forward + LN2 +
    // flags, timed as `stage`.
    ConvParams cp;
    std::memset(&cp, 0, sizeof cp);
    cp.X = act.X;
    cp.d = dec->d;
    cp.ntok = dec->ntok;
    cp.nbw = dec->nbw;
    cp.nwin = (int)n;
    cp.zero = dec->zero;
    auto post = [&](int l, int flags, int stage) -> hipError_t {
        if (!dec->dil[0]) return timed(dec, stage, s, [&] { return launch_tok(dec->D, dec->F, TOK_POST | MXF | flags, tp, n_tb, s); });
        tp.G = act.G[0];
        hipError_t e = timed(dec, PWD_STAGE_OUT_PROJ, s, [&] { return launch_tok(dec->D, dec->F, TOK_WO, tp, n_tb, s); });
        for (int j = 0; j < 3 && e == hipSuccess; ++j) {
            cp.Gin = act.G[j & 1];
            cp.Gout = act.G[(j + 1) & 1];
            cp.stream = dec->layers[l].conv[j];
            cp.bias = dec->layers[l].conv_b[j];
            cp.dil = dec->dil[j];
            e = timed(dec, PWD_STAGE_DILATED_CONV, s, [&] { return launch_conv(dec->D, j < 2, cp, n_tb, s); });
        }
        if (e != hipSuccess) return e;
        return timed(dec, stage, s, [&] { return launch_tok(dec->D, dec->F, TOK_FFN | flags, tp, n_tb, s); });
    };

    // round 0: embed (state D_0 = 0) and project layer 0
    tp.t = 0;
    set_qkv(0);
    HIP_OK(timed(dec, PWD_STAGE_EMBED_QKV, s, [&] { return launch_tok(dec->D, dec->F, TOK_EMBED | TOK_QKV | RES | MXF, tp, n_tb, s); }));
    for (int t = 0; t < dec->W; ++t) {
        const bool read_t = t >= dec->W - readouts;
        for (int l = 0; l < dec->L; ++l) {
            HIP_OK(timed(dec, PWD_STAGE_ATTENTION, s, [&] { return launch_attn(dec->dh, ap, (int)n, s); }));
            set_post(l);
            if (l + 1 < dec->L) {
                set_qkv(l + 1);
                HIP_OK(post(l, TOK_QKV, PWD_STAGE_POST_QKV));
            } else if (t + 1 < dec->W) {
                tp.t = t + 1;          // fold the next round's embedding into D_t
                set_qkv(0);
                // D_t for a readout goes to the Y buffer: each workgroup has read its own Y
                // tiles by then, and the next writer of Y is the next round's attention
                tp.state_out = read_t ? act.Y : nullptr;
                HIP_OK(post(l, TOK_EMBED | TOK_QKV | RES, PWD_STAGE_POST_EMBED_QKV));
                tp.state_out = nullptr;
                if (read_t) HIP_OK(readout(t - (dec->W - readouts), act.Y));
            } else {
                HIP_OK(post(l, 0, PWD_STAGE_POST));
            }
        }
    }
    HIP_OK(readout(readouts - 1, nullptr));
    return PWD_OK;
}

int decode_windows(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types, int64_t n,
                   float* d_logits, uint8_t* d_bits, void* hip_stream) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    return decode_impl(dec, d_meas, d_types, n, d_logits, d_bits, hip_stream, 1, handle_activations(dec));
}

int decode_windows_recurrent(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types, int64_t n,
                             float* d_logits, uint8_t* d_bits, void* hip_stream) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    return decode_impl(dec, d_meas, d_types, n, d_logits, d_bits, hip_stream, dec->d, handle_activations(dec));
}

int decode_windows_noalloc(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types, int64_t n,
                           float* d_logits, uint8_t* d_bits, void* hip_stream) {
    const int rc = check_batch(dec, d_meas, d_types, n, d_logits, d_bits);
    if (rc != PWD_OK || n == 0) return rc;
    Activations act{nullptr, nullptr, nullptr, {nullptr, nullptr}};
    if (dec->dtype != PWD_DTYPE_F32) {
        // the same token-block rounding as the handle's buffers: every launch's grid fits
        const int64_t gran = tok_block_granule();
        const int64_t n_tb = (n * dec->nbw + gran - 1) / gran * gran;
        size_t xb, qb, yb;
        const size_t need = activation_bytes(dec, n_tb, &xb, &qb, &yb);
        if (need > (size_t)PWD_NOALLOC_SCRATCH_BYTES)
            return fail(PWD_EBATCH, "%lld windows need %zu bytes of scratch; decode_windows_noalloc has %zu",
                        (long long)n, need, (size_t)PWD_NOALLOC_SCRATCH_BYTES);
        unsigned char* base = static_cast<unsigned char*>(dec->static_scratch);
        act.X = reinterpret_cast<float*>(base);
        act.QKV = reinterpret_cast<uint16_t*>(base + xb);
        act.Y = reinterpret_cast<uint16_t*>(base + xb + qb);
        if (dec->dil[0]) {
            act.G[0] = reinterpret_cast<uint16_t*>(base + xb + qb + yb);
            act.G[1] = reinterpret_cast<uint16_t*>(base + xb + qb + 2 * yb);
        }
    }
    return decode_impl(dec, d_meas, d_types, n, d_logits, d_bits, hip_stream, 1, act);
}

int decoder_detection_events(pwd_decoder* dec, const uint32_t* d_meas, const uint8_t* d_types,
                             int64_t n, uint32_t* d_events, void* hip_stream) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    if (n < 0) return fail(PWD_EINVAL, "negative n_windows");
    if (n > dec->max_windows) return fail(PWD_EBATCH, "n_windows %lld > max_windows %d", (long long)n, dec->max_windows);
    if (n == 0) return PWD_OK;
    if (!d_meas || !d_types || !d_events) return fail(PWD_EINVAL, "null buffer");
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    EventsParams p;
    p.in = syndrome_in(dec, d_meas, d_types, n);
    p.events = d_events;
    p.err = dec->err;
    HIP_OK(launch_events(p, static_cast<hipStream_t>(hip_stream)));
    return PWD_OK;
}

int decode_stream(pwd_decoder* dec, const uint32_t* d_stream, int64_t T, float* d_window_logits,
                  uint8_t* d_window_bits, float* d_window_probs, uint8_t* d_bit, float* d_prob, void* hip_stream) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    if (!d_stream || !d_bit) return fail(PWD_EINVAL, "null buffer");
    if (T <= 0) return fail(PWD_EINVAL, "stream of %lld rounds", (long long)T);
    const int64_t m = (T + dec->d - 1) / dec->d;
    if (m < 2 || m > dec->max_windows)
        return fail(PWD_EBATCH, "a stream of %lld rounds makes %lld windows; need 2..%d", (long long)T, (long long)m,
                    dec->max_windows);
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    StreamSplitParams sp;
    sp.stream = d_stream;
    sp.T = T;
    sp.m = (int)m;
    sp.d = dec->d;
    sp.W = dec->W;
    sp.b_left = dec->b_left;
    sp.words = dec->words;
    sp.meas = dec->stream_meas;
    sp.types = dec->stream_types;
    HIP_OK(timed(dec, PWD_STAGE_STREAM_SPLIT, s, [&] { return launch_stream_split(sp, s); }));
    float* logits = d_window_logits ? d_window_logits : dec->stream_logits;
    uint8_t* bits = d_window_bits ? d_window_bits : dec->stream_bits;
    const int rc = decode_windows(dec, dec->stream_meas, dec->stream_types, m, logits, bits, hip_stream);
    if (rc != PWD_OK) return rc;
    StreamCombineParams cp;
    cp.logits = logits;
    cp.bits = bits;
    cp.m = (int)m;
    cp.bit = d_bit;
    cp.prob = d_prob;
    cp.probs = d_window_probs;
    HIP_OK(timed(dec, PWD_STAGE_STREAM_COMBINE, s, [&] { return launch_stream_combine(cp, s); }));
    return PWD_OK;
}

int decoder_schedule(pwd_decoder* dec, int schedule) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    if (schedule != PWD_SCHEDULE_AUTO && schedule != PWD_SCHEDULE_LAYERS && schedule != PWD_SCHEDULE_RESIDENT)
        return fail(PWD_EINVAL, "schedule %d: need 0 (auto), 1 (layers) or 2 (resident)", schedule);
    if (schedule == PWD_SCHEDULE_RESIDENT && !dec->resident_ok)
        return fail(PWD_EUNSUPPORTED, "the resident schedule needs bf16, d_model 128, at most 64 tokens and 4 layers, "
                                      "heads of 16 or 32, feed-forward 4 d_model, no dilated convolutions or embedder block");
    dec->schedule = schedule;
    return PWD_OK;
}

int decoder_sync_status(pwd_decoder* dec, void* hip_stream) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    HIP_OK(hipStreamSynchronize(s));
    int flag = 0;
    HIP_OK(hipMemcpy(&flag, dec->err, sizeof(int), hipMemcpyDeviceToHost));
    if (flag) {
        HIP_OK(hipMemset(dec->err, 0, sizeof(int)));
        return fail(PWD_EDEVICE, "a window had an invalid type (> 2)");
    }
    return PWD_OK;
}

int decoder_profile(pwd_decoder* dec, int enable) {
    if (!dec) return fail(PWD_EINVAL, "null decoder");
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    for (auto& m : dec->marks) {
        HIP_OK(hipEventSynchronize(m.end));
        dec->spare.push_back(m.begin);
        dec->spare.push_back(m.end);
    }
    dec->marks.clear();
    dec->profiling = enable != 0;
    return PWD_OK;
}

int decoder_profile_read(pwd_decoder* dec, pwd_stage_times* out) {
    if (!dec || !out) return fail(PWD_EINVAL, "null decoder or output");
    DeviceGuard dg(dec->device);
    HIP_OK(dg.err);
    for (auto& m : dec->marks) {
        HIP_OK(hipEventSynchronize(m.end));
        float ms = 0.f;
        HIP_OK(hipEventElapsedTime(&ms, m.begin, m.end));
        out->ms[m.stage] += ms;
        out->launches[m.stage] += 1;
        dec->spare.push_back(m.begin);
        dec->spare.push_back(m.end);
    }
    dec->marks.clear();
    return PWD_OK;
}

}  // extern "C"
