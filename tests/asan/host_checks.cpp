// Host-side checks of the decoder library's C ABI, built with AddressSanitizer on the host
// code (the device code is unchanged): every configuration check, the blob parser on a valid
// blob and on corrupted and truncated copies (each in an allocation of exactly its length, so
// that a read past it is reported), the error strings, and the handle checks of the entry
// points. Exits non-zero on an unexpected return code; AddressSanitizer aborts on a memory error.
// Usage: host_checks <valid d=3 blob file>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/pwdec.h"

static int failures = 0;
#define EXPECT(cond, ...)                          \
    do {                                           \
        if (!(cond)) {                             \
            std::fprintf(stderr, "FAIL: " __VA_ARGS__); \
            std::fprintf(stderr, "\n");            \
            ++failures;                            \
        }                                          \
    } while (0)

static void touch_error() {
    const char* e = decoder_last_error();
    EXPECT(e != nullptr, "decoder_last_error returned null");
    if (e) (void)std::strlen(e);
}

static pwd_model_dims dims(int D, int L, int H, int r, int dt, int tok = 0, int emb = 0, int d0 = 0, int d1 = 0,
                           int d2 = 0) {
    pwd_model_dims m;
    std::memset(&m, 0, sizeof m);
    m.d_model = D;
    m.n_layers = L;
    m.n_heads = H;
    m.mlp_ratio = r;
    m.dtype = dt;
    m.token_set = tok;
    m.embedder = emb;
    m.conv_dilation[0] = d0;
    m.conv_dilation[1] = d1;
    m.conv_dilation[2] = d2;
    return m;
}

int main(int argc, char** argv) {
    if (argc != 2) {
        std::fprintf(stderr, "usage: %s blob\n", argv[0]);
        return 2;
    }
    // every geometry / dimension combination the checks distinguish, valid or not
    int checked = 0, valid = 0;
    for (int d = -1; d <= 67; d += 2)
        for (int wr : {0, 1, 2, 3, 4})
            for (int D : {0, 48, 64, 128, 256, 512})
                for (int H : {0, 1, 2, 4, 8, 16})
                    for (int dt : {-1, 0, 1, 2, 3})
                        for (int tok : {0, 1, 2}) {
                            const pwd_geometry g{d, wr * d - (wr == 4 ? 1 : 0), 16};
                            const pwd_model_dims m = dims(D, 2, H, 4, dt, tok, tok == 1 ? 1 : 0, tok == 1 ? 1 : 0,
                                                          tok == 1 ? 2 : 0, tok == 1 ? 4 : 0);
                            const int rc = decoder_validate_config(&g, &m);
                            EXPECT(rc == PWD_OK || rc == PWD_EINVAL || rc == PWD_EUNSUPPORTED,
                                   "validate d=%d W=%d D=%d H=%d dt=%d tok=%d: %d", d, g.window_rounds, D, H, dt, tok, rc);
                            if (rc == PWD_OK) {
                                ++valid;
                                EXPECT(decoder_blob_floats(&g, &m) > 0, "blob floats of a valid config");
                            } else {
                                touch_error();
                            }
                            ++checked;
                        }
    EXPECT(valid > 0 && valid < checked, "the sweep holds valid and invalid configurations");
    EXPECT(decoder_validate_config(nullptr, nullptr) == PWD_EINVAL, "null validate");
    touch_error();

    // the blob parser
    std::FILE* f = std::fopen(argv[1], "rb");
    if (!f) {
        std::fprintf(stderr, "cannot open %s\n", argv[1]);
        return 2;
    }
    std::vector<unsigned char> blob;
    unsigned char buf[65536];
    size_t n;
    while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) blob.insert(blob.end(), buf, buf + n);
    std::fclose(f);
    const pwd_geometry g3{3, 6, 4};
    const pwd_model_dims m3 = dims(64, 2, 4, 4, PWD_DTYPE_F32);
    EXPECT(decoder_validate_config(&g3, &m3) == PWD_OK, "d3 config");
    EXPECT(blob.size() == 64 + 4 * decoder_blob_floats(&g3, &m3), "d3 blob size %zu", blob.size());
    auto create = [&](const std::vector<unsigned char>& b) {
        unsigned char* copy = static_cast<unsigned char*>(std::malloc(b.size() ? b.size() : 1));
        if (!b.empty()) std::memcpy(copy, b.data(), b.size());
        pwd_decoder* h = nullptr;
        const int rc = decoder_create(&g3, &m3, copy, b.size(), &h);
        std::free(copy);
        if (rc == PWD_OK) {
            EXPECT(h != nullptr, "handle of a successful create");
            EXPECT(decoder_destroy(h) == PWD_OK, "destroy");
        } else {
            EXPECT(h == nullptr, "no handle on failure (%d)", rc);
            touch_error();
        }
        return rc;
    };
    // the valid blob: created on a device, or refused by the runtime where there is none
    const int rc_valid = create(blob);
    EXPECT(rc_valid == PWD_OK || rc_valid == PWD_EHIP || rc_valid == PWD_ENOMEM, "valid blob: %d", rc_valid);
    // every truncation of the header and a spread of truncations of the payload
    for (size_t len = 0; len < blob.size(); len += (len < 256 ? 1 : 997)) {
        const std::vector<unsigned char> t(blob.begin(), blob.begin() + len);
        const int rc = create(t);
        EXPECT(rc == PWD_EBLOB || rc == PWD_EINVAL, "truncated to %zu bytes: %d", len, rc);
    }
    // one word of the header changed at a time
    for (size_t w = 0; w < 16; ++w) {
        std::vector<unsigned char> c = blob;
        c[4 * w] ^= 0x5a;
        const int rc = create(c);
        EXPECT(rc != PWD_OK || w >= 14, "header word %zu corrupted: %d", w, rc);
    }
    std::vector<unsigned char> longer = blob;
    longer.insert(longer.end(), 4, 0);
    EXPECT(create(longer) == PWD_EBLOB, "blob with a trailing word");

    // entry points on a null handle
    EXPECT(decode_windows(nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr) == PWD_EINVAL, "decode null");
    EXPECT(decode_windows_recurrent(nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr) == PWD_EINVAL,
           "recurrent null");
    EXPECT(decoder_detection_events(nullptr, nullptr, nullptr, 0, nullptr, nullptr) == PWD_EINVAL, "events null");
    EXPECT(decoder_sync_status(nullptr, nullptr) == PWD_EINVAL, "sync null");
    EXPECT(decode_stream(nullptr, nullptr, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) == PWD_EINVAL,
           "stream null");
    EXPECT(decode_windows_noalloc(nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr) == PWD_EINVAL,
           "noalloc null");
    EXPECT(decoder_schedule(nullptr, 0) == PWD_EINVAL, "schedule null");
    EXPECT(decoder_profile(nullptr, 1) == PWD_EINVAL, "profile null");
    EXPECT(decoder_profile_read(nullptr, nullptr) == PWD_EINVAL, "profile read null");
    EXPECT(decoder_destroy(nullptr) == PWD_OK, "destroy null");
    touch_error();

    std::printf("host checks: %d configurations (%d valid), %zu-byte blob, %d failures\n", checked, valid,
                blob.size(), failures);
    return failures == 0 ? 0 : 1;
}
