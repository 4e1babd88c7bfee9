// Single-kernel entry points of the host build, for unit tests of one launch at a time.
#include "simt.h"
#include "kernels.h"

extern "C" int emu_attention(int dh, const uint16_t* qkv, uint16_t* y, int n_tokens, int npad, int nbw, int heads,
                             int nwin) {
    AttnParams p;
    p.QKV = qkv;
    p.Y = y;
    p.N = n_tokens;
    p.Npad = npad;
    p.nbw = nbw;
    p.H = heads;
    return (int)launch_attn(dh, p, nwin, nullptr);
}
