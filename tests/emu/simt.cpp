// simt.cpp - runtime of the host SIMT stand-in declared in simt.h: guard-paged allocations,
// the fiber scheduler with wavefront and workgroup barriers, LDS and its direct loads, and a
// fault handler that names what was running.
#include "simt.h"

#include <csignal>
#include <cstdarg>
#include <sys/mman.h>
#include <unistd.h>

#include <map>
#include <mutex>
#include <vector>

extern "C" char __start_emu_lds[], __stop_emu_lds[];

// One dynamic LDS allocation for every launch, in the LDS section like the static arrays.
static __attribute__((section("emu_lds"), aligned(256))) unsigned char g_dyn_lds[160 * 1024];

// x86-64 System V context switch: saves the callee-saved registers and the stack pointer of
// the running context in *save and resumes the one whose stack pointer is `to`.
extern "C" void emu_switch(void** save, void* to);
asm(R"(
.text
.globl emu_switch
.type emu_switch,@function
emu_switch:
    pushq %rbp
    pushq %rbx
    pushq %r12
    pushq %r13
    pushq %r14
    pushq %r15
    movq %rsp, (%rdi)
    movq %rsi, %rsp
    popq %r15
    popq %r14
    popq %r13
    popq %r12
    popq %rbx
    popq %rbp
    ret
.size emu_switch, .-emu_switch
)");

namespace emu {

Fiber* g_cur = nullptr;
emu_uint3 g_block_dim{1, 1, 1}, g_grid_dim{1, 1, 1};
Wave* g_waves = nullptr;
Group g_block;

namespace {

struct Alloc {
    char* base;       // the mapping
    size_t map_bytes;
    char* user;       // what hipMalloc returned
    size_t bytes;
};
std::map<uintptr_t, Alloc> g_allocs;   // by user pointer
std::vector<Alloc> g_freed;            // freed mappings stay PROT_NONE (use after free faults)
int g_errors = 0;
hipError_t g_last = hipSuccess;
const char* g_what = "";               // the running launch
uint64_t g_launch_no = 0;
void* g_sched_sp = nullptr;
Body g_body = nullptr;
void* g_ctx = nullptr;
std::vector<Fiber> g_fibers;
size_t g_page = 4096;
int g_trace = -1;

bool guard_at_start() {
    static int v = -1;
    if (v < 0) {
        const char* e = std::getenv("EMU_GUARD");
        v = e && std::strcmp(e, "start") == 0;
    }
    return v == 1;
}

const Alloc* find_alloc(uintptr_t a) {
    const Alloc* best = nullptr;
    for (auto& kv : g_allocs) {
        const Alloc& al = kv.second;
        if (a >= (uintptr_t)al.base && a < (uintptr_t)al.base + al.map_bytes) return &al;
    }
    return best;
}

void on_segv(int sig, siginfo_t* si, void*) {
    const uintptr_t a = (uintptr_t)si->si_addr;
    char buf[512];
    int n = snprintf(buf, sizeof buf, "\nEMU FAULT (signal %d) at %p during launch #%llu %s", sig, si->si_addr,
                     (unsigned long long)g_launch_no, g_what);
    if (g_cur)
        n += snprintf(buf + n, sizeof buf - n, " block %u thread %u", g_cur->bid.x, g_cur->tid.x);
    const Alloc* al = find_alloc(a);
    bool freed = false;
    if (!al)
        for (const Alloc& f : g_freed)
            if (a >= (uintptr_t)f.base && a < (uintptr_t)f.base + f.map_bytes) al = &f, freed = true;
    if (freed) n += snprintf(buf + n, sizeof buf - n, "; FREED");
    if (al)
        n += snprintf(buf + n, sizeof buf - n, "; allocation %p of %zu bytes, offset %lld", (void*)al->user,
                      al->bytes, (long long)(a - (uintptr_t)al->user));
    else
        n += snprintf(buf + n, sizeof buf - n, "; not near any live allocation");
    n += snprintf(buf + n, sizeof buf - n, "\n");
    (void)!write(2, buf, n);
    _exit(86);
}

void install_handler() {
    static bool done = false;
    if (done) return;
    done = true;
    static std::vector<char> alt(1 << 16);
    stack_t ss{};
    ss.ss_sp = alt.data();
    ss.ss_size = alt.size();
    sigaltstack(&ss, nullptr);
    struct sigaction sa{};
    sa.sa_sigaction = on_segv;
    sa.sa_flags = SA_SIGINFO | SA_ONSTACK;
    sigaction(SIGSEGV, &sa, nullptr);
    sigaction(SIGBUS, &sa, nullptr);
    g_page = (size_t)sysconf(_SC_PAGESIZE);
}

[[noreturn]] void fiber_main() {
    g_body(g_ctx);
    Fiber* f = g_cur;
    f->done = true;
    emu_switch(&f->sp, g_sched_sp);
    __builtin_trap();
}

constexpr size_t STACK_BYTES = 512 * 1024;

void init_fiber(Fiber& f) {
    if (!f.stack) {
        // stack with a guard page below it
        char* m = (char*)mmap(nullptr, STACK_BYTES + g_page, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS, -1, 0);
        if (m == MAP_FAILED) {
            report("fiber stack allocation failed");
            std::abort();
        }
        mprotect(m, g_page, PROT_NONE);
        f.stack = m;
        f.stack_bytes = STACK_BYTES + g_page;
    }
    uintptr_t top = ((uintptr_t)f.stack + f.stack_bytes) & ~(uintptr_t)15;
    void** sp = (void**)top;
    *--sp = nullptr;                            // fake return address of fiber_main
    *--sp = (void*)&fiber_main;                 // emu_switch returns here
    for (int i = 0; i < 6; ++i) *--sp = nullptr;   // rbp rbx r12 r13 r14 r15
    f.sp = sp;
    f.done = false;
    f.wait_g = nullptr;
    f.xset = 0;
    f.xseq = 0;
    f.npend = 0;
}

void release(Group& g) {
    g.arrived = 0;
    ++g.gen;
}

}  // namespace

void report(const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    fprintf(stderr, "EMU ERROR: %s (launch #%llu %s, block %u thread %u)\n", buf, (unsigned long long)g_launch_no,
            g_what, g_cur ? g_cur->bid.x : 0u, g_cur ? g_cur->tid.x : 0u);
    ++g_errors;
}
int errors() { return g_errors; }

void barrier(Group& g) {
    const uint64_t my = g.gen;
    if (++g.arrived >= g.alive) {
        release(g);
        return;
    }
    Fiber* f = g_cur;
    f->wait_g = &g;
    f->wait_gen = my;
    emu_switch(&f->sp, g_sched_sp);
    f->wait_g = nullptr;
}

void check_tags() {
    Wave& w = g_waves[g_cur->wave];
    const uint64_t mine = w.tag[g_cur->xset][g_cur->lane];
    const int n = w.bar.alive + 0;
    (void)n;
    for (int l = 0; l < 64; ++l) {
        if (l >= (int)g_block_dim.x - 64 * g_cur->wave) break;
        const Fiber& other = g_fibers[64 * g_cur->wave + l];
        if (other.done) continue;
        if (w.tag[g_cur->xset][l] != mine) {
            report("lanes %d and %d of wavefront %d meet at different cross-lane operations (%llx, %llx)",
                   g_cur->lane, l, g_cur->wave, (unsigned long long)mine, (unsigned long long)w.tag[g_cur->xset][l]);
            return;
        }
    }
}

char* lds_base() { return __start_emu_lds; }
size_t lds_bytes() { return (size_t)(__stop_emu_lds - __start_emu_lds); }
void* dyn_smem() { return g_dyn_lds; }

void lds_dma(int bytes, uint32_t voff, const void* sbase, uint32_t m0) {
    Fiber* f = g_cur;
    if (f->npend >= 64) {
        report("more than 64 direct LDS loads outstanding in one lane");
        f->npend = 0;
    }
    Fiber::Dma& d = f->pend[f->npend++];
    d.lds = m0 + (uint32_t)(f->lane * bytes);
    d.bytes = bytes;
    std::memcpy(d.data, static_cast<const char*>(sbase) + voff, (size_t)bytes);   // faults on a bad source
    if ((size_t)d.lds + (size_t)bytes > lds_bytes()) report("direct LDS load writes past LDS (offset %u)", d.lds);
}

void waitcnt() {
    Fiber* f = g_cur;
    for (int i = 0; i < f->npend; ++i) {
        const Fiber::Dma& d = f->pend[i];
        if ((size_t)d.lds + (size_t)d.bytes <= lds_bytes()) std::memcpy(lds_base() + d.lds, d.data, (size_t)d.bytes);
    }
    f->npend = 0;
}

void run_grid(const char* what, dim3 grid, dim3 block, size_t smem, Body body, void* ctx) {
    install_handler();
    if (g_trace < 0) g_trace = std::getenv("EMU_TRACE") != nullptr;
    ++g_launch_no;
    g_what = what;
    if (g_trace) fprintf(stderr, "emu launch #%llu %s grid %u block %u smem %zu\n", (unsigned long long)g_launch_no,
                         what, grid.x, block.x, smem);
    const int nthreads = (int)(block.x * block.y * block.z);
    if (grid.y != 1 || grid.z != 1 || block.y != 1 || block.z != 1 || nthreads < 1 || nthreads > 1024 ||
        smem > sizeof g_dyn_lds) {
        report("unsupported launch shape");
        g_last = hipErrorInvalidValue;
        return;
    }
    g_body = body;
    g_ctx = ctx;
    g_block_dim = {block.x, 1, 1};
    g_grid_dim = {grid.x, 1, 1};
    const int nwaves = (nthreads + 63) / 64;
    std::vector<Wave> waves(nwaves);
    g_waves = waves.data();
    if ((int)g_fibers.size() < nthreads) g_fibers.resize(nthreads);
    for (uint32_t b = 0; b < grid.x; ++b) {
        std::memset(lds_base(), 0xff, lds_bytes());   // NaN pattern: unwritten LDS is visible
        g_block = Group{};
        g_block.alive = nthreads;
        for (int w = 0; w < nwaves; ++w) {
            waves[w].bar = Group{};
            waves[w].bar.alive = std::min(64, nthreads - 64 * w);
        }
        for (int t = 0; t < nthreads; ++t) {
            Fiber& f = g_fibers[t];
            init_fiber(f);
            f.tid = {(uint32_t)t, 0, 0};
            f.bid = {b, 0, 0};
            f.lane = t & 63;
            f.wave = t >> 6;
        }
        int left = nthreads;
        while (left > 0) {
            bool ran = false;
            for (int t = 0; t < nthreads; ++t) {
                Fiber& f = g_fibers[t];
                if (f.done) continue;
                if (f.wait_g && f.wait_g->gen == f.wait_gen) continue;
                g_cur = &f;
                emu_switch(&g_sched_sp, f.sp);
                g_cur = nullptr;
                ran = true;
                if (f.done) {
                    --left;
                    if (f.npend) report("direct LDS loads still pending at the end of work-item %d", t);
                    Group* gs[2] = {&waves[f.wave].bar, &g_block};
                    for (Group* g : gs)
                        if (--g->alive > 0 && g->arrived >= g->alive) release(*g);
                }
            }
            if (!ran) {
                report("deadlock: work-items wait at barriers that the others never reach");
                g_last = hipErrorLaunchFailure;
                return;
            }
        }
    }
    g_waves = nullptr;
    g_what = "";
}

}  // namespace emu

using namespace emu;

// Each allocation sits in the middle of GUARD bytes of inaccessible address space on either
// side, so an access that misses it by up to GUARD faults instead of landing in another buffer.
constexpr size_t GUARD = (size_t)8 << 30;

hipError_t hipMalloc(void** p, size_t bytes) {
    install_handler();
    if (!p) return hipErrorInvalidValue;
    const size_t data_pages = (bytes + g_page - 1) / g_page + (bytes == 0);
    const size_t map_bytes = 2 * GUARD + data_pages * g_page;
    char* m = (char*)mmap(nullptr, map_bytes, PROT_NONE, MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE, -1, 0);
    if (m == MAP_FAILED) return hipErrorOutOfMemory;
    char* data = m + GUARD;
    if (mprotect(data, data_pages * g_page, PROT_READ | PROT_WRITE) != 0) return hipErrorOutOfMemory;
    // against the inaccessible space after the end (16-byte aligned: sizes round up to 16), or
    // at the start of the first page with EMU_GUARD=start
    const size_t rb = (bytes + 15) & ~(size_t)15;
    char* user = guard_at_start() ? data : data + data_pages * g_page - rb;
    std::memset(user, 0xa5, bytes);   // garbage, as fresh device memory may hold
    g_allocs[(uintptr_t)user] = Alloc{m, map_bytes, user, bytes};
    *p = user;
    return hipSuccess;
}

hipError_t hipFree(void* p) {
    if (!p) return hipSuccess;
    auto it = g_allocs.find((uintptr_t)p);
    if (it == g_allocs.end()) return hipErrorInvalidValue;
    mprotect(it->second.base, it->second.map_bytes, PROT_NONE);   // never unmapped: use after free faults
    g_freed.push_back(it->second);
    g_allocs.erase(it);
    return hipSuccess;
}

hipError_t hipMemcpy(void* dst, const void* src, size_t bytes, hipMemcpyKind) {
    if (bytes) std::memmove(dst, src, bytes);
    return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind k, hipStream_t) {
    return hipMemcpy(dst, src, bytes, k);
}
hipError_t hipMemset(void* p, int v, size_t bytes) {
    if (bytes) std::memset(p, v, bytes);
    return hipSuccess;
}
hipError_t hipMemsetAsync(void* p, int v, size_t bytes, hipStream_t) { return hipMemset(p, v, bytes); }
hipError_t hipGetDevice(int* d) {
    *d = 0;
    return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipGetLastError() {
    const hipError_t e = g_last;
    g_last = hipSuccess;
    return e;
}
const char* hipGetErrorString(hipError_t e) {
    switch (e) {
        case hipSuccess: return "no error";
        case hipErrorInvalidValue: return "invalid argument";
        case hipErrorOutOfMemory: return "out of memory";
        default: return "launch failure";
    }
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipDeviceSynchronize() { return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t* e) {
    *e = reinterpret_cast<hipEvent_t>(new char[1]);
    return hipSuccess;
}
hipError_t hipEventDestroy(hipEvent_t e) {
    delete[] reinterpret_cast<char*>(e);
    return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
    *ms = 0.f;
    return hipSuccess;
}
hipError_t hipFuncSetAttribute(const void*, hipFuncAttribute, int) { return hipSuccess; }
hipError_t hipGetSymbolAddress(void** p, const void* symbol) {
    *p = const_cast<void*>(symbol);
    return hipSuccess;
}

// Entry points for the Python side of the tests: "device" buffers and the error count.
extern "C" {
void* emu_malloc(size_t bytes) {
    void* p = nullptr;
    return hipMalloc(&p, bytes) == hipSuccess ? p : nullptr;
}
void emu_free(void* p) { (void)hipFree(p); }
int emu_errors(void) { return emu::errors(); }
// The i-th live allocation (in address order): its pointer and size; returns 0 past the last.
int emu_allocation(int i, void** ptr, size_t* bytes) {
    for (auto& kv : g_allocs)
        if (i-- == 0) {
            *ptr = kv.second.user;
            *bytes = kv.second.bytes;
            return 1;
        }
    return 0;
}
}
