// CPU emulation of the subset of HIP used by paper_1710_09854_amd/csrc/gspar.hip.
//
// TEST INFRASTRUCTURE: lets the unchanged library source be compiled with g++ (optionally with
// AddressSanitizer) and run on the host, so kernel indexing and solver logic can be checked on a
// machine without a GPU. Each launch runs its workgroups one after another. The threads of a
// workgroup are fibers on the calling host thread, each with its own stack, switched cooperatively
// at the points where a GPU thread can wait for another: __syncthreads, the per-wave exchanges
// behind shuffles and ballots, wave barriers and s_sleep. A fiber runs until it reaches such a
// point; a barrier releases when every fiber of its group that has not returned has arrived, and
// the fiber that completes it runs on first, so the others observe its later writes only after
// their own next switch. EMU_SHUFFLE=1 picks the next fiber at random instead of round robin
// (seeded per launch and workgroup, and by EMU_SHUFFLE_SEED), which changes which lanes run first after each barrier and exposes
// reads of shared state that no barrier separates from another lane's write. __shared__ variables
// become static storage, shared by the fibers of the running workgroup. Because workgroups never
// overlap, inter-workgroup waits (the look-back) always find their predecessors finished.
#pragma once
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <chrono>
#include <condition_variable>
#include <dlfcn.h>
#include <sys/mman.h>
#include <mutex>
#include <random>
#include <functional>
#include <memory>
#include <thread>
#include <vector>
#if defined(__SANITIZE_ADDRESS__)
#include <sanitizer/common_interface_defs.h>
#endif

#define __global__
#define __device__
#define __host__
#define __shared__ static
#define __forceinline__ inline
#define __noinline__ __attribute__((noinline))
#define __launch_bounds__(...)

using std::max;
using std::min;

struct dim3 {
  unsigned x, y, z;
  dim3(unsigned a = 1, unsigned b = 1, unsigned c = 1) : x(a), y(b), z(c) {}
};
struct uint3e {
  unsigned x = 0, y = 0, z = 0;
};
struct float4 {
  float x, y, z, w;
};
inline float4 make_float4(float a, float b, float c, float d) { return float4{a, b, c, d}; }

typedef int hipError_t;
typedef void* hipStream_t;
typedef void* hipEvent_t;
enum { hipSuccess = 0 };
inline hipError_t hipGetLastError() { return hipSuccess; }
// device symbols are host storage here: the symbol's address is the variable's own
#define __align__(n) alignas(n)
#define HIP_SYMBOL(x) (&(x))
inline hipError_t hipGetDevice(int* d) { *d = 0; return hipSuccess; }
inline hipError_t hipGetSymbolAddress(void** p, const void* sym) { *p = const_cast<void*>(sym); return hipSuccess; }
inline hipError_t hipEventCreate(hipEvent_t* e) { *e = nullptr; return hipSuccess; }
inline hipError_t hipEventDestroy(hipEvent_t) { return hipSuccess; }
inline hipError_t hipEventRecord(hipEvent_t, hipStream_t = nullptr) { return hipSuccess; }
inline hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
inline hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) { *ms = 0.f; return hipSuccess; }

namespace emu {
// A barrier among the fibers of a group: `expected` drops when a member returns from the kernel.
struct Bar {
  unsigned expected = 0, arrived = 0;
  unsigned long gen = 0;
};
struct Wave {
  uint64_t buf[64];
  Bar bar;
};
struct Block {
  Bar bar;
  std::vector<Wave> waves;
};
struct Fiber {
  void* sp = nullptr;
  char* stack = nullptr;  // lowest usable address (a guard page lies below it)
  unsigned tid = 0;
  bool done = false;
  unsigned long nsync = 0;
};
inline constexpr size_t kFiberStack = size_t(1) << 20;
inline Block* tl_block = nullptr;
inline uint3e tl_tid, tl_bid, tl_bdim, tl_gdim;
// Stall diagnostics: each lane records the call site and count of its last block barrier.
struct LaneTrace {
  std::atomic<const void*> site{nullptr};
  std::atomic<unsigned long> n{0};
  std::atomic<unsigned> block{0};
};
inline LaneTrace g_trace[1024];
inline bool g_shuffle = getenv("EMU_SHUFFLE") && atoi(getenv("EMU_SHUFFLE")) != 0;
// EMU_SHUFFLE_SEED varies the random schedules between runs
inline unsigned g_shuffle_seed = getenv("EMU_SHUFFLE_SEED") ? (unsigned)atoi(getenv("EMU_SHUFFLE_SEED")) : 0u;
inline unsigned long g_launches = 0;
inline std::minstd_rand g_rng;

// scheduler state of the running launch (launches come from one host thread at a time)
inline std::vector<Fiber> g_fibers;
inline unsigned g_nfib = 0, g_cur = 0, g_live = 0;
inline std::vector<unsigned> g_alive, g_slot;  // the fibers that have not returned, and where each sits
inline void* g_main_sp = nullptr;
inline void (*g_body)(void*) = nullptr;
inline void* g_body_arg = nullptr;
#if defined(__SANITIZE_ADDRESS__)
inline const void* g_main_bottom = nullptr;
inline size_t g_main_size = 0;
inline bool g_from_main = false;
#endif

// Saves the callee-saved registers and the stack pointer of the running context in *save and
// resumes the context whose stack pointer is `load` (System V x86-64).
extern "C" __attribute__((visibility("hidden"))) void emu_fiber_switch(void** save, void* load);
asm(".text\n"
    ".globl emu_fiber_switch\n.hidden emu_fiber_switch\n.type emu_fiber_switch,@function\n.p2align 4\n"
    "emu_fiber_switch:\n"
    "  pushq %rbp\n  pushq %rbx\n  pushq %r12\n  pushq %r13\n  pushq %r14\n  pushq %r15\n"
    "  movq %rsp, (%rdi)\n  movq %rsi, %rsp\n"
    "  popq %r15\n  popq %r14\n  popq %r13\n  popq %r12\n  popq %rbx\n  popq %rbp\n  ret\n"
    ".size emu_fiber_switch,.-emu_fiber_switch\n");

inline void enter(unsigned next) {
  g_cur = next;
  tl_tid.x = g_fibers[next].tid;
}
// Switches from the running fiber to fiber `next` (the running one if `next` equals it).
inline void switch_to(unsigned next) {
  const unsigned from = g_cur;
  if (next == from) return;
  enter(next);
#if defined(__SANITIZE_ADDRESS__)
  void* fake = nullptr;
  __sanitizer_start_switch_fiber(&fake, g_fibers[next].stack, kFiberStack);
  emu_fiber_switch(&g_fibers[from].sp, g_fibers[next].sp);
  __sanitizer_finish_switch_fiber(fake, nullptr, nullptr);
#else
  emu_fiber_switch(&g_fibers[from].sp, g_fibers[next].sp);
#endif
}
// The next fiber that has not returned: round robin after the running one, or a random one.
inline unsigned pick() {
  if (g_shuffle) return g_alive[g_rng() % g_live];
  unsigned t = g_cur;
  do t = (t + 1) % g_nfib;
  while (g_fibers[t].done);
  return t;
}
inline void yield() { switch_to(pick()); }
inline void release(Bar& b) {
  b.arrived = 0;
  ++b.gen;
}
inline unsigned long g_events = 0;  // barrier arrivals and returns from the kernel
[[noreturn]] void deadlock();
inline void bar_wait(Bar& b) {
  const unsigned long gen = b.gen;
  ++g_events;
  if (++b.arrived == b.expected) {
    release(b);
    if (g_shuffle && (g_rng() & 3) == 0) yield();  // let others run first now and then
    return;
  }
  // Every fiber that has not returned gets the processor between two resumptions of this one
  // (round robin; at random, with overwhelming probability within 64 rounds): when this fiber
  // resumes that often with no arrival or return anywhere, every fiber waits and none can release.
  unsigned long seen = g_events, idle = 0;
  while (b.gen == gen) {
    yield();
    if (g_events != seen) {
      seen = g_events;
      idle = 0;
    } else if (++idle > (g_shuffle ? 64u * g_live : 2u)) {
      deadlock();
    }
  }
}
// A member returns from the kernel: the barrier no longer waits for it.
inline void bar_drop(Bar& b) {
  --b.expected;
  if (b.arrived != 0 && b.arrived == b.expected) release(b);
}
}  // namespace emu

#define threadIdx (emu::tl_tid)
#define blockIdx (emu::tl_bid)
#define blockDim (emu::tl_bdim)
#define gridDim (emu::tl_gdim)

__attribute__((noinline)) inline void __syncthreads() {
  auto& tr = emu::g_trace[emu::tl_tid.x];
  tr.site.store(__builtin_return_address(0));
  tr.n.fetch_add(1);
  ++emu::g_fibers[emu::g_cur].nsync;
  emu::bar_wait(emu::tl_block->bar);
}
inline void __threadfence() { std::atomic_thread_fence(std::memory_order_seq_cst); }

namespace emu {
inline Wave& wave() { return tl_block->waves[tl_tid.x / 64]; }
inline int lane() { return tl_tid.x % 64; }
template <class T>
inline T xchg(T v, int src) {
  static_assert(sizeof(T) <= 8, "lane exchange of at most 8 bytes");
  Wave& w = wave();
  uint64_t b = 0;
  std::memcpy(&b, &v, sizeof(T));
  w.buf[lane()] = b;
  emu::bar_wait(w.bar);
  uint64_t r = w.buf[src & 63];
  emu::bar_wait(w.bar);
  T out;
  std::memcpy(&out, &r, sizeof(T));
  return out;
}
}  // namespace emu

template <class T>
inline T __shfl(T v, int src, int = 64) { return emu::xchg(v, src); }
template <class T>
inline T __shfl_xor(T v, int mask, int = 64) { return emu::xchg(v, emu::lane() ^ mask); }
template <class T>
inline T __shfl_down(T v, unsigned delta, int = 64) {
  int l = emu::lane();
  return emu::xchg(v, l + (int)delta < 64 ? l + (int)delta : l);
}
template <class T>
inline T __shfl_up(T v, unsigned delta, int = 64) {
  int l = emu::lane();
  T r = emu::xchg(v, l >= (int)delta ? l - (int)delta : l);
  return r;
}
inline unsigned long long __ballot(int pred) {
  emu::Wave& w = emu::wave();
  w.buf[emu::lane()] = pred ? 1 : 0;
  emu::bar_wait(w.bar);
  unsigned long long m = 0;
  for (int i = 0; i < 64; ++i) m |= (unsigned long long)(w.buf[i] != 0) << i;
  emu::bar_wait(w.bar);
  return m;
}
inline void __builtin_amdgcn_wave_barrier() { emu::bar_wait(emu::wave().bar); }
inline unsigned __builtin_amdgcn_mbcnt_lo(unsigned m, unsigned acc) {
  const int l = emu::lane();
  return acc + (unsigned)__builtin_popcount(l >= 32 ? m : (m & ((1u << l) - 1u)));
}
inline unsigned __builtin_amdgcn_mbcnt_hi(unsigned m, unsigned acc) {
  const int l = emu::lane();
  return acc + (unsigned)__builtin_popcount(l < 32 ? 0u : (m & (l == 63 ? 0x7fffffffu : ((1u << (l - 32)) - 1u))));
}
// v_perm_b32: byte i of the result is chosen by byte i of sel from the eight bytes of {s0, s1}
// (s1 the low word): 0-7 a byte, 8-11 the sign bit of byte 1, 3, 5 or 7 replicated, 12 zero,
// 13 and above 0xFF.
inline unsigned __builtin_amdgcn_perm(unsigned s0, unsigned s1, unsigned sel) {
  const unsigned long long in = ((unsigned long long)s0 << 32) | s1;
  unsigned r = 0;
  for (int i = 0; i < 4; ++i) {
    const unsigned s = (sel >> (8 * i)) & 0xFF;
    unsigned b;
    if (s >= 13) b = 0xFF;
    else if (s == 12) b = 0x00;
    else if (s >= 8) b = ((in >> (16 * (s - 8) + 15)) & 1) ? 0xFF : 0x00;
    else b = (unsigned)(in >> (8 * s)) & 0xFF;
    r |= b << (8 * i);
  }
  return r;
}
// v_sad_u8: the sum over the four bytes of |a_i - b_i|, plus c.
inline unsigned __builtin_amdgcn_sad_u8(unsigned a, unsigned b, unsigned c) {
  unsigned r = c;
  for (int i = 0; i < 4; ++i) {
    const int x = (int)((a >> (8 * i)) & 0xFF), y = (int)((b >> (8 * i)) & 0xFF);
    r += (unsigned)(x > y ? x - y : y - x);
  }
  return r;
}
struct uint4 {
  unsigned x, y, z, w;
};
inline uint4 make_uint4(unsigned x, unsigned y, unsigned z, unsigned w) { return uint4{x, y, z, w}; }
inline int __popc(unsigned v) { return __builtin_popcount(v); }
inline int __popcll(unsigned long long v) { return __builtin_popcountll(v); }
inline void __builtin_amdgcn_s_sleep(int) { emu::yield(); }
inline void __builtin_amdgcn_sched_barrier(int) {}
inline void __builtin_amdgcn_s_waitcnt(int) {}
inline unsigned __float_as_uint(float f) {
  unsigned u;
  std::memcpy(&u, &f, 4);
  return u;
}
inline int __ffsll(unsigned long long v) { return __builtin_ffsll((long long)v); }

template <class T, class U>
inline T atomicAdd(T* p, U v) { return __atomic_fetch_add(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U>
inline T atomicOr(T* p, U v) { return __atomic_fetch_or(p, (T)v, __ATOMIC_SEQ_CST); }
template <class T, class U>
inline T atomicMax(T* p, U v) {
  T old = __atomic_load_n(p, __ATOMIC_SEQ_CST);
  while (old < (T)v && !__atomic_compare_exchange_n(p, &old, (T)v, false, __ATOMIC_SEQ_CST, __ATOMIC_SEQ_CST)) {
  }
  return old;
}
#define __HIP_MEMORY_SCOPE_AGENT 0
namespace emu {
// EMU_HIDE_STATUS=1: loads of look-back status words (values with either of the top two bits
// set) read as "not yet published", which drives the look-back into its fallback path.
inline bool g_hide_status = getenv("EMU_HIDE_STATUS") && atoi(getenv("EMU_HIDE_STATUS")) != 0;
template <class T>
inline T atomic_load_emu(T* p) {
  T v = __atomic_load_n(p, __ATOMIC_SEQ_CST);
  if constexpr (sizeof(T) == 8) {
    if (g_hide_status && ((uint64_t)v >> 62) != 0) return (T)0;
  }
  return v;
}
}  // namespace emu
#define __hip_atomic_load(p, order, scope) emu::atomic_load_emu(p)
#define __hip_atomic_store(p, v, order, scope) __atomic_store_n((p), (v), __ATOMIC_SEQ_CST)

namespace emu {
// No fiber of the running workgroup can proceed (a lane waits at a barrier its partners never
// reach): report where each lane passed its last block barrier and stop.
[[noreturn]] inline void deadlock() {
  Dl_info info;
  dladdr((void*)&__syncthreads, &info);
  fprintf(stderr, "EMU DEADLOCK in block %u: lanes (tid block-barriers passed site-offset):\n", tl_bid.x);
  for (unsigned t = 0; t < g_nfib; ++t)
    if (!g_fibers[t].done)
      fprintf(stderr, "  %u %lu 0x%lx\n", t, g_fibers[t].nsync,
              (unsigned long)((const char*)g_trace[t].site.load() - (const char*)info.dli_fbase));
  fflush(stderr);
  abort();
}

// A new fiber starts here: it runs the kernel for its lane, leaves its barriers and passes control
// to another fiber that has not returned, or back to the launch when it was the last.
[[noreturn]] inline void fiber_start() {
#if defined(__SANITIZE_ADDRESS__)
  const void* from_bottom = nullptr;
  size_t from_size = 0;
  __sanitizer_finish_switch_fiber(nullptr, &from_bottom, &from_size);
  if (g_from_main) {  // the launch's own stack, for the switch back at the end
    g_main_bottom = from_bottom;
    g_main_size = from_size;
    g_from_main = false;
  }
#endif
  const unsigned me = g_cur;
  g_body(g_body_arg);
  Fiber& f = g_fibers[me];
  f.done = true;
  --g_live;
  ++g_events;
  const unsigned last = g_alive[g_live];  // swap the returned fiber out of the live list
  g_alive[g_slot[me]] = last;
  g_slot[last] = g_slot[me];
  bar_drop(tl_block->bar);
  bar_drop(tl_block->waves[f.tid / 64].bar);
  void* dead = nullptr;
  if (g_live == 0) {
#if defined(__SANITIZE_ADDRESS__)
    __sanitizer_start_switch_fiber(nullptr, g_main_bottom, g_main_size);
#endif
    emu_fiber_switch(&dead, g_main_sp);
  } else {
    const unsigned next = pick();
    enter(next);
#if defined(__SANITIZE_ADDRESS__)
    __sanitizer_start_switch_fiber(nullptr, g_fibers[next].stack, kFiberStack);
#endif
    emu_fiber_switch(&dead, g_fibers[next].sp);
  }
  __builtin_unreachable();
}

// Stacks for up to n fibers, kept for later launches: 1 MiB each above a guard page, mapped on
// demand.
inline void ensure_fibers(unsigned n) {
  while (g_fibers.size() < n) {
    const size_t page = 4096;
    char* m = (char*)mmap(nullptr, kFiberStack + page, PROT_READ | PROT_WRITE,
                          MAP_PRIVATE | MAP_ANONYMOUS | MAP_NORESERVE | MAP_STACK, -1, 0);
    if (m == MAP_FAILED) {
      fprintf(stderr, "EMU: cannot map a fiber stack\n");
      abort();
    }
    mprotect(m, page, PROT_NONE);
    Fiber f;
    f.stack = m + page;
    g_fibers.push_back(f);
  }
}

// Runs the workgroups of a launch one after another, each as block.x fibers on this thread.
template <class K, class... A>
void launch(K kernel, dim3 grid, dim3 block, A... args) {
  const unsigned nb = grid.x * grid.y * grid.z;
  const unsigned nt = block.x;
  ensure_fibers(nt);
  ++g_launches;
  Block blk;
  // EMU_STALL_SECONDS: a launch still running after that long reports each lane's last block
  // barrier and exits (a lane that loops without reaching a barrier)
  std::mutex mu;
  std::condition_variable cv;
  bool finished = false;
  const int stall_s = getenv("EMU_STALL_SECONDS") ? atoi(getenv("EMU_STALL_SECONDS")) : 0;
  std::thread watchdog;
  if (stall_s > 0) {
    watchdog = std::thread([&] {
      std::unique_lock<std::mutex> lk(mu);
      if (cv.wait_for(lk, std::chrono::seconds(stall_s), [&] { return finished; })) return;
      Dl_info info;
      dladdr((void*)&__syncthreads, &info);
      fprintf(stderr, "EMU STALL: launch of %u x %u; lanes (tid block count site-offset):\n", nb, nt);
      for (unsigned t = 0; t < nt; ++t) {
        const void* site = g_trace[t].site.load();
        fprintf(stderr, "  %u %u %lu 0x%lx\n", t, g_trace[t].block.load(), g_trace[t].n.load(),
                (unsigned long)((const char*)site - (const char*)info.dli_fbase));
      }
      fflush(stderr);
      _exit(3);
    });
  }
  auto body = [&]() { kernel(args...); };
  g_body = [](void* p) { (*static_cast<decltype(body)*>(p))(); };
  g_body_arg = &body;
  bool divergent = false;
  for (unsigned b = 0; b < nb && !divergent; ++b) {
    blk.bar = Bar{nt, 0, 0};
    blk.waves.assign((nt + 63) / 64, Wave{});
    for (unsigned w = 0; w < blk.waves.size(); ++w) blk.waves[w].bar.expected = std::min(64u, nt - 64 * w);
    tl_block = &blk;
    tl_bid.x = b % grid.x;
    tl_bid.y = (b / grid.x) % grid.y;
    tl_bdim.x = block.x;
    tl_gdim.x = grid.x;
    tl_gdim.y = grid.y;
    g_rng.seed(1234567u + b + 7919u * (unsigned)g_launches + 104729u * g_shuffle_seed);
    for (unsigned t = 0; t < nt; ++t) {
      Fiber& f = g_fibers[t];
      f.tid = t;
      f.done = false;
      f.nsync = 0;
      g_trace[t].block.store(b);
      // initial frame: six zero registers, then fiber_start as the return address, then an unused
      // slot, so that fiber_start begins with the stack aligned as after a call
      void** top = (void**)(f.stack + kFiberStack);
      top[-1] = nullptr;
      top[-2] = (void*)&fiber_start;
      for (int r = 3; r <= 8; ++r) top[-r] = nullptr;
      f.sp = (void*)(top - 8);
    }
    g_nfib = g_live = nt;
    g_alive.resize(nt);
    g_slot.resize(nt);
    for (unsigned t = 0; t < nt; ++t) g_alive[t] = g_slot[t] = t;
    enter(0);
#if defined(__SANITIZE_ADDRESS__)
    void* fake = nullptr;
    g_from_main = true;
    __sanitizer_start_switch_fiber(&fake, g_fibers[0].stack, kFiberStack);
    emu_fiber_switch(&g_main_sp, g_fibers[0].sp);
    __sanitizer_finish_switch_fiber(fake, nullptr, nullptr);
#else
    emu_fiber_switch(&g_main_sp, g_fibers[0].sp);
#endif
    // every thread of a workgroup must pass the same number of block barriers
    for (unsigned u = 1; u < nt; ++u)
      if (g_fibers[u].nsync != g_fibers[0].nsync) {
        fprintf(stderr, "EMU DIVERGENT BARRIERS: block %u lane 0 passed %lu, lane %u passed %lu\n", b,
                g_fibers[0].nsync, u, g_fibers[u].nsync);
        divergent = true;
        break;
      }
  }
  {
    std::lock_guard<std::mutex> lk(mu);
    finished = true;
  }
  cv.notify_all();
  if (watchdog.joinable()) watchdog.join();
  if (divergent) abort();
}
}  // namespace emu

#define hipLaunchKernelGGL(kernel, grid, block, shmem, stream, ...) emu::launch(kernel, grid, block, __VA_ARGS__)
#define HIP_KERNEL_NAME(...) __VA_ARGS__
