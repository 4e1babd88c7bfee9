// Shared device-side definitions of the decoder's HIP kernels (gfx950 / CDNA4).
//
// Layouts. The bf16 path keeps every activation in the register layout of the MFMA
// instruction v_mfma_f32_16x16x32_bf16, with tokens along the MFMA column (lane % 16) and
// features along rows, so a GEMM is computed transposed (Out^T = W^T In^T) and one
// GEMM's accumulator feeds the next GEMM's B operand without a shuffle:
//   * C fragment of a 16x16 tile: lane l holds rows 4*(l/16)+i, i = 0..3, of column l%16.
//   * B fragment of a 32-deep k-step: lane l holds column l%16 and 8 k values at slots
//     kslot(l/16, i) = i < 4 ? 4g+i : 16+4g+(i-4). Two C tiles stacked along k (rows
//     0-15 and 16-31) are exactly that B fragment, so "C -> B" is a bf16 pack.
//   * A fragment (weights, rows = output features, k = input features): lane l holds row
//     l%16 and the same 8 k slots.
// Tokens are grouped in blocks of 16 (one MFMA column block). A window of N = d*d-1
// stabilizers is padded to Npad = 16*ceil(N/16) tokens; padding tokens carry finite values
// that never reach real tokens (attention masks them as keys, the readout skips them).
//
// In HBM (per token block tb, all "fragment-major" so a wave moves 1 KB contiguous):
//   X   fp32 [tb][D/16][64][4]   residual stream / recurrent state, C fragments
//   QKV bf16 [tb][3][D/32][64][8] B fragments of Q, K and V (features h*dh.. of head h)
//   Y   bf16 [tb][D/32][64][8]   attention output, B fragments
//   weights bf16 [D_out/16][D_in/32][64][8] A fragments of W^T
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

#define PWD_DEV static __device__ __forceinline__

// Per-window type codes (App. A.1.1).
#define WIN_INITIAL 0
#define WIN_BULK 1
#define WIN_FINAL 2

// A wavefront-uniform pointer, pinned to scalar registers.
template <typename T>
PWD_DEV const T* uniform_ptr(const T* p) {
    const uint64_t v = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return reinterpret_cast<const T*>(((uint64_t)hi << 32) | lo);
}

// 32-bit LDS address of a __shared__ location.
template <typename T>
PWD_DEV uint32_t lds_addr(T* p) {
    return (uint32_t)reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) T*)p);
}

// One direct global->LDS load of 1 KB: lane l copies bytes [16 l, 16 l + 16) of the
// wavefront-uniform `src` to LDS address `lds` + 16 l. Inline assembly, because the compiler's
// wait-count pass treats a pending direct-to-LDS builtin as outstanding LDS traffic and then
// waits for every LDS read before each use; callers await completion with s_waitcnt vmcnt.
// The memory clobber keeps the load in program order relative to other memory accesses.
// The compiler cannot see the operands of inline assembly when it inserts the wait states the
// hardware requires, and a vector instruction that writes an SGPR (v_readfirstlane, which
// uniform_ptr becomes when the address was computed in VGPRs) must be followed by 5 of them
// before a vector memory instruction reads that SGPR as its address; otherwise the load uses
// the register's previous contents. LDS_DMA_GUARD provides them (and the one an SALU write of
// M0 needs before the load reads it).
#define LDS_DMA_GUARD "s_nop 4\n\t"
PWD_DEV void lds_load_1k(const void* src, uint32_t lds, int lane) {
    asm volatile(LDS_DMA_GUARD "global_load_lds_dwordx4 %0, %1" :: "v"((uint32_t)lane * 16), "s"(src), "{m0}"(lds)
                 : "memory");
}

PWD_DEV int kslot(int g, int i) { return i < 4 ? 4 * g + i : 16 + 4 * g + (i - 4); }

PWD_DEV f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
PWD_DEV f32x4 mfma16x16x16(bf16x4 a, bf16x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Two C tiles (k rows 0-15 and 16-31 of a k-step) -> one bf16 B fragment.
PWD_DEV bf16x8 pack_b(f32x4 lo, f32x4 hi) {
    bf16x8 r;
    r[0] = (__bf16)lo[0]; r[1] = (__bf16)lo[1]; r[2] = (__bf16)lo[2]; r[3] = (__bf16)lo[3];
    r[4] = (__bf16)hi[0]; r[5] = (__bf16)hi[1]; r[6] = (__bf16)hi[2]; r[7] = (__bf16)hi[3];
    return r;
}

// Reductions across the four 16-lane groups of a wavefront (lanes l, l^16, l^32, l^48 -- the
// four row groups of an MFMA C fragment's column) with the gfx950 lane-swap instructions, in the
// vector ALU rather than through LDS: v_permlane32_swap exchanges the upper half of one register
// with the lower half of another, so with both holding v each lane sees v of lane l^32; then
// v_permlane16_swap does the same for lane l^16. Every lane gets the same result.
PWD_DEV float swap32(float v, float& other) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    other = __uint_as_float(r[1]);
    return __uint_as_float(r[0]);
}
PWD_DEV float swap16(float v, float& other) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    other = __uint_as_float(r[1]);
    return __uint_as_float(r[0]);
}
PWD_DEV float group_sum(float v) {
    float o;
    const float a = swap32(v, o);
    v = a + o;
    const float b = swap16(v, o);
    return b + o;
}
PWD_DEV float group_max(float v) {
    float o;
    const float a = swap32(v, o);
    v = fmaxf(a, o);
    const float b = swap16(v, o);
    return fmaxf(b, o);
}
// the value of lane l % 16 (row 0 of a C fragment's column) in every lane
PWD_DEV float row0_broadcast(float v) {
    float o;
    const float a = swap16(v, o);   // lanes of rows 0 and 1 now hold row 0's value
    return swap32(a, o);            // and the upper half receives the lower half
}

// Detection events at window round t, one 32-stabilizer word (Sec. 2.2: a detector is the
// parity of two consecutive measurements of one stabilizer; App. A.1.1: zero padding replaces
// the missing buffer of the initial and final windows; the initial window's first core round
// is compared with the all-zero state): event_from takes the words of rows t (prev) and t + 1
// (cur), event_word reads them from the window's rows meas [W+1][words].
PWD_DEV uint32_t event_from(uint32_t prev, uint32_t cur, int t, int type, int b_left, int d) {
    if (type == WIN_INITIAL) {
        if (t < b_left) return 0u;
        if (t == b_left) prev = 0u;
    } else if (type == WIN_FINAL) {
        if (t >= b_left + d) return 0u;
    }
    return cur ^ prev;
}
PWD_DEV uint32_t event_word(const uint32_t* __restrict__ meas, int words, int t, int w,
                            int type, int b_left, int d) {
    return event_from(meas[t * words + w], meas[(t + 1) * words + w], t, type, b_left, d);
}
