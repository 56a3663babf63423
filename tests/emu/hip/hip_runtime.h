// CPU emulation of the subset of HIP used by paper_1710_09854_amd/csrc/gspar.hip.
//
// TEST INFRASTRUCTURE: lets the unchanged library source be compiled with g++ (optionally with
// AddressSanitizer) and run on the host, so kernel indexing and solver logic can be checked on a
// machine without a GPU. Each launch runs its workgroups one after another; the threads of a
// workgroup are real host threads, synchronised by a barrier for __syncthreads and by per-wave
// barriers for cross-lane operations (shuffles, ballots). __shared__ variables become static
// storage, shared by the threads of the running workgroup. Because workgroups never overlap,
// inter-workgroup waits (the look-back) always find their predecessors finished.
#pragma once
#include <algorithm>
#include <atomic>
#include <barrier>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <chrono>
#include <dlfcn.h>
#include <mutex>
#include <random>
#include <functional>
#include <memory>
#include <thread>
#include <vector>

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
struct Wave {
  uint64_t buf[64];
  std::unique_ptr<std::barrier<>> bar;
};
struct Block {
  std::unique_ptr<std::barrier<>> bar;
  std::vector<Wave> waves;
};
inline thread_local Block* tl_block = nullptr;
inline thread_local uint3e tl_tid, tl_bid, tl_bdim, tl_gdim;
// Stall diagnostics: each lane records the call site and count of its last block barrier.
struct LaneTrace {
  std::atomic<const void*> site{nullptr};
  std::atomic<unsigned long> n{0};
  std::atomic<unsigned> block{0};
};
inline LaneTrace g_trace[1024];
inline thread_local unsigned long tl_nsync = 0;
inline thread_local std::minstd_rand tl_rng;
inline int g_jitter_us = getenv("EMU_JITTER_US") ? atoi(getenv("EMU_JITTER_US")) : 0;
}  // namespace emu

#define threadIdx (emu::tl_tid)
#define blockIdx (emu::tl_bid)
#define blockDim (emu::tl_bdim)
#define gridDim (emu::tl_gdim)

__attribute__((noinline)) inline void __syncthreads() {
  auto& tr = emu::g_trace[emu::tl_tid.x];
  tr.site.store(__builtin_return_address(0));
  tr.n.fetch_add(1);
  ++emu::tl_nsync;
  emu::tl_block->bar->arrive_and_wait();
  // optional jitter: every lane but 0 may lag after a barrier, exposing reads of shared state that
  // are not separated from lane 0's next write by a barrier
  if (emu::g_jitter_us > 0 && emu::tl_tid.x != 0 && (emu::tl_rng() & 3) == 0)
    std::this_thread::sleep_for(std::chrono::microseconds(emu::tl_rng() % emu::g_jitter_us));
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
  w.bar->arrive_and_wait();
  uint64_t r = w.buf[src & 63];
  w.bar->arrive_and_wait();
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
  w.bar->arrive_and_wait();
  unsigned long long m = 0;
  for (int i = 0; i < 64; ++i) m |= (unsigned long long)(w.buf[i] != 0) << i;
  w.bar->arrive_and_wait();
  return m;
}
inline void __builtin_amdgcn_wave_barrier() { emu::wave().bar->arrive_and_wait(); }
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
inline void __builtin_amdgcn_s_sleep(int) { std::this_thread::yield(); }
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
// One host thread per lane of the workgroup, reused for every workgroup of the launch. Between
// workgroups all threads meet at `between`; the workgroup's barriers are then rebuilt, since
// threads that returned early dropped out of them.
template <class K, class... A>
void launch(K kernel, dim3 grid, dim3 block, A... args) {
  const unsigned nb = grid.x * grid.y * grid.z;
  const unsigned nt = block.x;
  Block blk;
  auto rebuild = [&] {
    blk.bar = std::make_unique<std::barrier<>>(nt);
    blk.waves.clear();
    blk.waves.resize((nt + 63) / 64);
    for (auto& w : blk.waves) w.bar = std::make_unique<std::barrier<>>(std::min<unsigned>(64, nt));
  };
  rebuild();
  std::barrier<> between(nt);
  std::atomic<bool> finished{false};
  const int stall_s = getenv("EMU_STALL_SECONDS") ? atoi(getenv("EMU_STALL_SECONDS")) : 0;
  std::thread watchdog;
  if (stall_s > 0) {
    watchdog = std::thread([&] {
      auto t0 = std::chrono::steady_clock::now();
      while (!finished.load()) {
        std::this_thread::sleep_for(std::chrono::milliseconds(50));
        if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(stall_s)) {
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
        }
      }
    });
  }
  std::vector<unsigned long> nsync(nt);
  std::atomic<int> divergent{0};
  std::vector<std::thread> th;
  th.reserve(nt);
  for (unsigned t = 0; t < nt; ++t) {
    th.emplace_back([&, t] {
      for (unsigned b = 0; b < nb; ++b) {
        g_trace[t].block.store(b);
        tl_block = &blk;
        tl_tid.x = t;
        tl_bid.x = b % grid.x;
        tl_bid.y = (b / grid.x) % grid.y;
        tl_bdim.x = block.x;
        tl_gdim.x = grid.x;
        tl_gdim.y = grid.y;
        tl_rng.seed(1234567u * (t + 1) + b);
        tl_nsync = 0;
        kernel(args...);
        nsync[t] = tl_nsync;
        // a thread leaving early must not block its workgroup's remaining barriers
        blk.bar->arrive_and_drop();
        blk.waves[t / 64].bar->arrive_and_drop();
        between.arrive_and_wait();
        if (t == 0) {
          // every thread of a workgroup must pass the same number of block barriers
          for (unsigned u = 1; u < nt; ++u)
            if (nsync[u] != nsync[0]) {
              fprintf(stderr, "EMU DIVERGENT BARRIERS: block %u lane 0 passed %lu, lane %u passed %lu\n", b,
                      nsync[0], u, nsync[u]);
              divergent.store(1);
              break;
            }
          rebuild();
        }
        between.arrive_and_wait();
      }
    });
  }
  for (auto& x : th) x.join();
  finished.store(true);
  if (watchdog.joinable()) watchdog.join();
  if (divergent.load()) abort();
}
}  // namespace emu

#define hipLaunchKernelGGL(kernel, grid, block, shmem, stream, ...) emu::launch(kernel, grid, block, __VA_ARGS__)
#define HIP_KERNEL_NAME(...) __VA_ARGS__
