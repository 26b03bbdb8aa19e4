// Host stand-in for the HIP runtime header: just enough to compile the planner
// (paper_2506_05433_amd/csrc/pg_plan.hpp) as ordinary C++ for the tests. A workgroup is
// run as `threads` std::threads, __syncthreads() is a std::barrier, and __shared__
// variables become function-local statics shared by those threads. Blocks of a grid run
// one after another. Built with AddressSanitizer by tests/test_plan_host.py.
#pragma once
#include <algorithm>
#include <barrier>
#include <thread>
#include <vector>

#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static

struct HostDim3 {
  unsigned x = 0, y = 1, z = 1;
};
inline thread_local HostDim3 threadIdx;
inline thread_local HostDim3 blockIdx;
inline HostDim3 blockDim;
inline std::barrier<>* g_block_barrier = nullptr;

inline void __syncthreads() { g_block_barrier->arrive_and_wait(); }
inline int atomicOr(int* p, int v) { return __atomic_fetch_or(p, v, __ATOMIC_SEQ_CST); }
using std::max;
using std::min;

// Runs body() as `grid` workgroups of `threads` threads each: `threads` host threads step
// through the workgroups together, meeting at a barrier between two workgroups.
template <class F>
void host_launch(unsigned grid, unsigned threads, F body) {
  blockDim.x = threads;
  std::barrier<> bar((std::ptrdiff_t)threads);
  g_block_barrier = &bar;
  std::vector<std::thread> ts;
  ts.reserve(threads);
  for (unsigned t = 0; t < threads; ++t)
    ts.emplace_back([&body, &bar, t, grid] {
      threadIdx.x = t;
      for (unsigned b = 0; b < grid; ++b) {
        blockIdx.x = b;
        body();
        bar.arrive_and_wait();
      }
    });
  for (auto& th : ts) th.join();
}
