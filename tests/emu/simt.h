// simt.h - a host (x86-64) stand-in for the HIP runtime and the gfx950 device features the
// decoder's kernels use, so that the library's own kernel sources can be compiled for the CPU
// and run there under memory checks. Test infrastructure only: nothing in the library loads it.
//
// Execution model. A launch runs its workgroups one after another; each work-item is a fiber
// with its own stack, and fibers switch only at synchronisation points:
//   * __syncthreads: every live work-item of the workgroup arrives;
//   * cross-lane operations (MFMA, shuffles, readfirstlane, ballot): every live lane of the
//     wavefront arrives, each having posted its operands to the wavefront's exchange slots.
// So the kernel code runs unmodified, lane by lane, with the same data exchange as on the GPU.
// Lanes of a wavefront that disagree on the sequence of cross-lane operations, or a barrier
// that not every work-item reaches, end in a reported deadlock.
//
// Memory checks. hipMalloc places every allocation against a PROT_NONE guard page (after its
// end, or before its start with EMU_GUARD=start), so an access past it faults on the host with
// the allocation, the kernel, the workgroup and the work-item named. LDS (static __shared__
// arrays and the dynamic allocation) lives in one linker section, is filled with 0xff (a NaN
// pattern) before every workgroup, and the direct global->LDS loads land only when the issuing
// lane waits for its vector memory counter, so LDS read before its wait shows up as NaN.
#pragma once
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <tuple>
#include <type_traits>
#include <utility>

// ---- qualifiers
#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __align__(n) __attribute__((aligned(n)))
#define __shared__ static __attribute__((section("emu_lds")))

// ---- runtime types
typedef enum hipError_t {
    hipSuccess = 0,
    hipErrorInvalidValue = 1,
    hipErrorOutOfMemory = 2,
    hipErrorLaunchFailure = 719,
} hipError_t;
typedef enum hipMemcpyKind {
    hipMemcpyHostToHost = 0,
    hipMemcpyHostToDevice = 1,
    hipMemcpyDeviceToHost = 2,
    hipMemcpyDeviceToDevice = 3,
    hipMemcpyDefault = 4
} hipMemcpyKind;
typedef enum hipFuncAttribute { hipFuncAttributeMaxDynamicSharedMemorySize = 8 } hipFuncAttribute;
struct ihipStream_t;
typedef ihipStream_t* hipStream_t;
struct ihipEvent_t;
typedef ihipEvent_t* hipEvent_t;

struct dim3 {
    uint32_t x, y, z;
    constexpr dim3(uint32_t x_ = 1, uint32_t y_ = 1, uint32_t z_ = 1) : x(x_), y(y_), z(z_) {}
};
struct emu_uint3 {
    uint32_t x, y, z;
};

hipError_t hipMalloc(void** p, size_t bytes);
template <class T>
hipError_t hipMalloc(T** p, size_t bytes) { return hipMalloc(reinterpret_cast<void**>(p), bytes); }
hipError_t hipFree(void* p);
hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind);
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind, hipStream_t = nullptr);
hipError_t hipMemset(void* p, int v, size_t bytes);
hipError_t hipMemsetAsync(void* p, int v, size_t bytes, hipStream_t = nullptr);
hipError_t hipGetDevice(int* d);
hipError_t hipSetDevice(int d);
hipError_t hipGetLastError();
const char* hipGetErrorString(hipError_t e);
hipError_t hipStreamSynchronize(hipStream_t);
hipError_t hipDeviceSynchronize();
hipError_t hipEventCreate(hipEvent_t* e);
hipError_t hipEventDestroy(hipEvent_t e);
hipError_t hipEventRecord(hipEvent_t e, hipStream_t = nullptr);
hipError_t hipEventSynchronize(hipEvent_t e);
hipError_t hipEventElapsedTime(float* ms, hipEvent_t a, hipEvent_t b);
hipError_t hipFuncSetAttribute(const void*, hipFuncAttribute, int);
hipError_t hipGetSymbolAddress(void** p, const void* symbol);
#define HIP_SYMBOL(x) (&(x))

// ---- device-side vector types (identical to the kernels' own typedefs)
typedef __bf16 emu_bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 emu_bf16x4 __attribute__((ext_vector_type(4)));
typedef float emu_f32x4 __attribute__((ext_vector_type(4)));

namespace emu {

struct Group {
    uint64_t gen = 0;
    int arrived = 0;
    int alive = 0;
};

struct Wave {
    Group bar;
    alignas(16) unsigned char slot[2][64][64];   // double-buffered exchange, 64 bytes per lane
    uint64_t tag[2][64];                         // (kind, sequence number) each lane posted
};

struct Fiber {
    void* sp = nullptr;
    void* stack = nullptr;
    size_t stack_bytes = 0;
    emu_uint3 tid{0, 0, 0}, bid{0, 0, 0};
    int lane = 0, wave = 0, xset = 0;
    uint32_t xseq = 0;   // cross-lane operations this lane has posted
    bool done = false;
    Group* wait_g = nullptr;
    uint64_t wait_gen = 0;
    // direct global->LDS loads issued by this lane and not yet waited for
    struct Dma { uint32_t lds; int bytes; unsigned char data[16]; };
    Dma pend[64];
    int npend = 0;
};

extern Fiber* g_cur;
extern emu_uint3 g_block_dim, g_grid_dim;
extern Wave* g_waves;
extern Group g_block;

void barrier(Group& g);
void check_tags();
inline void wave_sync() {
    barrier(g_waves[g_cur->wave].bar);
    check_tags();
}
inline void block_sync() { barrier(g_block); }

// Posts this lane's operand of a cross-lane operation of the given kind; after the wavefront
// barrier every lane checks that all lanes posted the same operation (a lane that skips or
// adds one would otherwise silently pair with another operation).
template <class T>
inline void xput(const T& v, uint32_t kind = sizeof(T)) {
    static_assert(sizeof(T) <= 64, "exchange slot");
    Wave& w = g_waves[g_cur->wave];
    std::memcpy(w.slot[g_cur->xset][g_cur->lane], &v, sizeof(T));
    w.tag[g_cur->xset][g_cur->lane] = ((uint64_t)kind << 32) | g_cur->xseq++;
}
template <class T>
inline T xget(int lane) {
    T r;
    std::memcpy(&r, g_waves[g_cur->wave].slot[g_cur->xset][lane & 63], sizeof(T));
    return r;
}
inline void xdone() { g_cur->xset ^= 1; }
template <class T>
inline T exchange(const T& v, int src_lane) {
    xput(v);
    wave_sync();
    const T r = xget<T>(src_lane);
    xdone();
    return r;
}

char* lds_base();
size_t lds_bytes();
void* dyn_smem();
void lds_dma(int bytes, uint32_t voff, const void* sbase, uint32_t m0);
void waitcnt();
void report(const char* fmt, ...);
int errors();

// Launch: workgroups in order, each as block.x fibers that run k(args...).
using Body = void (*)(void*);
void run_grid(const char* what, dim3 grid, dim3 block, size_t smem, Body body, void* ctx);

template <class K, class Tup>
struct LaunchCtx {
    K k;
    Tup args;
};
template <class K, class Tup>
void call_kernel(void* c) {
    auto* x = static_cast<LaunchCtx<K, Tup>*>(c);
    std::apply(x->k, x->args);
}
template <class K, class... A>
void launch(const char* what, K k, dim3 grid, dim3 block, size_t smem, hipStream_t, A&&... args) {
    using Tup = std::tuple<std::decay_t<A>...>;
    LaunchCtx<K, Tup> ctx{k, Tup(std::forward<A>(args)...)};
    run_grid(what, grid, block, smem, &call_kernel<K, Tup>, &ctx);
}

}  // namespace emu

#define threadIdx (emu::g_cur->tid)
#define blockIdx (emu::g_cur->bid)
#define blockDim (emu::g_block_dim)
#define gridDim (emu::g_grid_dim)

inline void __syncthreads() { emu::block_sync(); }

template <class T>
inline T __shfl_xor(T v, int mask, int width = 64) {
    const int lane = emu::g_cur->lane, src = lane ^ mask;
    return emu::exchange(v, (src & ~(width - 1)) == (lane & ~(width - 1)) ? src : lane);
}
template <class T>
inline T __shfl(T v, int src, int width = 64) {
    const int lane = emu::g_cur->lane;
    return emu::exchange(v, (lane & ~(width - 1)) + (src & (width - 1)));
}

template <class A, class B>
inline std::common_type_t<A, B> min(A a, B b) { return a < b ? a : b; }
template <class A, class B>
inline std::common_type_t<A, B> max(A a, B b) { return a < b ? b : a; }
inline float rsqrtf(float x) { return 1.0f / std::sqrt(x); }
inline unsigned __float_as_uint(float f) { unsigned u; std::memcpy(&u, &f, 4); return u; }
inline float __uint_as_float(unsigned u) { float f; std::memcpy(&f, &u, 4); return f; }

template <class T>
inline T atomicOr(T* p, T v) {
    const T old = *p;
    *p = old | v;
    return old;
}

// ---- the AMDGPU builtins the kernels call (their sources are renamed emu_amdgcn_*)
template <class T>
inline T emu_amdgcn_readfirstlane(T v) { return emu::exchange(v, 0); }
inline uint64_t emu_amdgcn_ballot_w64(bool b) {
    emu::xput<int>(b ? 1 : 0);
    emu::wave_sync();
    uint64_t m = 0;
    for (int l = 0; l < 64; ++l)
        if (emu::xget<int>(l)) m |= 1ull << l;
    emu::xdone();
    return m;
}
inline float emu_amdgcn_exp2f(float x) { return std::exp2(x); }
inline float emu_amdgcn_rcpf(float x) { return 1.0f / x; }
typedef unsigned int emu_u32x2 __attribute__((ext_vector_type(2)));
// v_permlane32_swap / v_permlane16_swap: the upper half (odd 16-lane rows) of the first operand
// swaps with the lower half (even rows) of the second; returns (first, second) after the swap.
inline emu_u32x2 emu_permlane_swap(unsigned v, unsigned s, int span) {
    struct P { unsigned v, s; };
    emu::xput(P{v, s}, 100 + span);
    emu::wave_sync();
    const int lane = emu::g_cur->lane;
    const bool upper = (lane / span) & 1;
    const P mine = emu::xget<P>(lane), peer = emu::xget<P>(upper ? lane - span : lane + span);
    emu::xdone();
    // upper lanes of the first operand take the second operand of the lower peer; lower lanes of
    // the second operand take the first operand of the upper peer
    return upper ? emu_u32x2{peer.s, mine.s} : emu_u32x2{mine.v, peer.v};
}
inline emu_u32x2 emu_amdgcn_permlane32_swap(unsigned v, unsigned s, bool, bool) { return emu_permlane_swap(v, s, 32); }
inline emu_u32x2 emu_amdgcn_permlane16_swap(unsigned v, unsigned s, bool, bool) { return emu_permlane_swap(v, s, 16); }
inline void emu_amdgcn_sched_group_barrier(int, int, int) {}
inline void emu_amdgcn_sched_barrier(int) {}

// v_mfma_f32_16x16x{32,16}_bf16: D[row][col] = C + sum_k A[row][k] B[k][col]. Lane l holds
// A row l % 16 and B column l % 16 with the k values of lane group l / 16 in its register
// elements; the lane's D elements are rows 4 (l / 16) + i of column l % 16. The k order within
// a lane group does not matter for the sum as long as A and B share it, which both kernels
// and the host-side weight layout do.
template <class V, int NV>
inline emu_f32x4 emu_mfma_16x16(V a, V b, emu_f32x4 c) {
    struct AB { V a, b; };
    emu::xput(AB{a, b});
    emu::wave_sync();
    const int lane = emu::g_cur->lane, col = lane & 15, g = lane >> 4;
    AB bcol[4];
    for (int gg = 0; gg < 4; ++gg) bcol[gg] = emu::xget<AB>(col + 16 * gg);
    emu_f32x4 d;
    for (int i = 0; i < 4; ++i) {
        const int row = 4 * g + i;
        double s = 0.0;
        for (int gg = 0; gg < 4; ++gg) {
            const AB ar = emu::xget<AB>(row + 16 * gg);
            for (int k = 0; k < NV; ++k) s += (double)(float)ar.a[k] * (double)(float)bcol[gg].b[k];
        }
        d[i] = c[i] + (float)s;
    }
    emu::xdone();
    return d;
}
inline emu_f32x4 emu_amdgcn_mfma_f32_16x16x32_bf16(emu_bf16x8 a, emu_bf16x8 b, emu_f32x4 c, int, int, int) {
    return emu_mfma_16x16<emu_bf16x8, 8>(a, b, c);
}
inline emu_f32x4 emu_amdgcn_mfma_f32_16x16x16bf16_1k(emu_bf16x4 a, emu_bf16x4 b, emu_f32x4 c, int, int, int) {
    return emu_mfma_16x16<emu_bf16x4, 4>(a, b, c);
}

// ---- 8-bit floating point (MXFP8 path)
typedef int emu_i32x8 __attribute__((ext_vector_type(8)));
inline float emu_amdgcn_fmed3f(float a, float b, float c) { return std::fmax(std::fmin(a, b), std::fmin(std::fmax(a, b), c)); }
// E4M3 (OCP FP8): value of a code, NaN for S.1111.111
inline double emu_e4m3_value(unsigned code) {
    const double sign = (code & 0x80) ? -1.0 : 1.0;
    const int e = (code >> 3) & 15, m = code & 7;
    if (e == 15 && m == 7) return NAN;
    return e == 0 ? sign * std::ldexp((double)m, -9) : sign * std::ldexp(1.0 + m / 8.0, e - 7);
}
// v_cvt_pk_fp8_f32 as measured on gfx950: round to nearest, ties to even, on the E4M3 grid
// extended by 480; results past 448 (480 and beyond) give the NaN code, no saturation.
inline unsigned emu_e4m3_code(float f) {
    const unsigned sign = std::signbit(f) ? 0x80u : 0u;
    const double a = std::fabs((double)f);
    if (std::isnan(a)) return sign | 0x7fu;
    if (a < std::ldexp(1.0, -6)) return sign | (unsigned)std::nearbyint(std::ldexp(a, 9));
    int e;
    std::frexp(a, &e);
    int E = e - 1;
    if (E > 8) return sign | 0x7fu;
    int q = (int)std::nearbyint((std::ldexp(a, -E) - 1.0) * 8.0);
    if (q == 8) { q = 0; ++E; }
    if (E > 8 || (E == 8 && q == 7)) return sign | 0x7fu;
    return sign | (unsigned)(((E + 7) << 3) | q);
}
inline int emu_amdgcn_cvt_pk_fp8_f32(float a, float b, int old, bool hi) {
    const unsigned w = emu_e4m3_code(a) | (emu_e4m3_code(b) << 8);
    return hi ? (int)(((unsigned)old & 0xffffu) | (w << 16)) : (int)(((unsigned)old & 0xffff0000u) | w);
}
// v_mfma_scale_f32_16x16x128_f8f6f4 with E4M3 operands, as measured on gfx950: byte e of lane
// group g of A (row l % 16) pairs with byte e of lane group g of B (column l % 16); those bytes
// form K block kb = 2 (e / 16) + g / 2, whose E8M0 scales (byte opsel of the scale operand)
// come from lane row + 16 kb of A and lane col + 16 kb of B.
inline emu_f32x4 emu_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(emu_i32x8 a, emu_i32x8 b, emu_f32x4 c, int cbsz,
                                                             int blgp, int opsel_a, int sa, int opsel_b, int sb) {
    if (cbsz != 0 || blgp != 0) emu::report("mfma_scale: only E4M3 operands are emulated");
    struct Op { emu_i32x8 v; unsigned s; };
    // two exchanges (a slot holds 64 bytes): every lane's A operand and scale, then B's
    const int lane = emu::g_cur->lane, col = lane & 15, g = lane >> 4;
    Op A[64], Bv[64];
    emu::xput(Op{a, ((unsigned)sa >> (8 * opsel_a)) & 0xffu});
    emu::wave_sync();
    for (int l = 0; l < 64; ++l) A[l] = emu::xget<Op>(l);
    emu::xdone();
    emu::xput(Op{b, ((unsigned)sb >> (8 * opsel_b)) & 0xffu}, 1);
    emu::wave_sync();
    for (int l = 0; l < 64; ++l) Bv[l] = emu::xget<Op>(l);
    emu::xdone();
    emu_f32x4 d;
    for (int i = 0; i < 4; ++i) {
        const int row = 4 * g + i;
        double s = 0.0;
        for (int gg = 0; gg < 4; ++gg) {
            const Op& ar = A[row + 16 * gg];
            const Op& bc = Bv[col + 16 * gg];
            for (int e = 0; e < 32; ++e) {
                const int kb = 2 * (e / 16) + gg / 2;
                const unsigned ca = ((unsigned)ar.v[e / 4] >> (8 * (e % 4))) & 0xffu;
                const unsigned cb = ((unsigned)bc.v[e / 4] >> (8 * (e % 4))) & 0xffu;
                const double xa = std::ldexp(1.0, (int)A[row + 16 * kb].s - 127);
                const double xb = std::ldexp(1.0, (int)Bv[col + 16 * kb].s - 127);
                s += emu_e4m3_value(ca) * emu_e4m3_value(cb) * xa * xb;
            }
        }
        d[i] = c[i] + (float)s;
    }
    return d;
}

// ---- the kernels' inline assembly, as rewritten by the source transformation
inline uint32_t emu_lds_off(const void* p) {
    const char* c = static_cast<const char*>(p);
    if (c < emu::lds_base() || c >= emu::lds_base() + emu::lds_bytes())
        emu::report("lds_addr of a pointer outside LDS: %p", p);
    return (uint32_t)(c - emu::lds_base());
}
inline void emu_lds_dma(int bytes, uint32_t voff, const void* sbase, uint32_t m0) {
    emu::lds_dma(bytes, voff, sbase, m0);
}
inline void emu_waitcnt_vm(int) { emu::waitcnt(); }
