// Dispatch order of a segment's tasks.
//
// The attention kernel gives each XCD a contiguous range of the dispatch
// order, and an XCD holds a few dozen tasks at once that all stream K/V
// tiles through its own L2.  Two tasks share L2 lines only if they read the
// same tile at nearly the same time, which in practice means their tile lists
// are equal and they start together.  Tasks built in row order rarely are:
// under a multi-dimensional window, query blocks with equal KV lists sit a
// grid stride apart, and tasks with shorter lists drift ahead of the others.
// Sorting the tasks of each (batch, head) by their first and then their last
// KV tile puts equal lists next to each other, so they are dispatched
// together, finish together, and their successors start together.  The sort
// is stable: tasks with equal keys keep their row order.  Every task still
// computes exactly what it computed before, so results do not change.
#include <hipcub/hipcub.hpp>

#include "bsa_internal.h"

namespace bsa {

namespace {

// Key of task t: (bh, first tile, last tile) packed into key_bits bits.
// Entries past the device task count get the largest key, so the stable
// sort leaves the real tasks in front.
__global__ __launch_bounds__(256) void task_key_kernel(OrderArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.ntasks) return;
  const int64_t nt = a.ntasks_dev ? *a.ntasks_dev : a.ntasks;
  uint64_t key = a.key_bits >= 64 ? ~0ull : ((1ull << a.key_bits) - 1);
  if (t < nt) {
    const Task tk = a.tasks[t];
    uint64_t first = 0, last = 0;
    if (tk.tile_end > tk.tile_begin) {
      first = (uint32_t)a.tile_kv[tk.tile_begin];
      last = (uint32_t)a.tile_kv[tk.tile_end - 1];
    }
    key = ((uint64_t)(uint32_t)tk.bh << (2 * a.tile_bits)) | (first << a.tile_bits) | last;
  }
  a.keys_in[t] = key;
  a.idx_in[t] = (int32_t)t;
}

// The tasks themselves in dispatch order, so the kernel reads its task with
// no indirection (tasks without Split-K partners only: the merge finds the
// partial states of a row's pieces next to each other in row order).
__global__ __launch_bounds__(256) void task_gather_kernel(OrderArgs a) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= a.ntasks) return;
  a.tasks_out[t] = a.tasks[a.order[t]];
}

}  // namespace

int task_order_key_bits(int64_t nbh, int64_t ntiles, int* tile_bits) {
  auto bits_for = [](int64_t n) {  // bits of the largest index n - 1, at least 1
    int b = 1;
    while (b < 63 && (int64_t(1) << b) < n) ++b;
    return b;
  };
  *tile_bits = bits_for(ntiles);
  return bits_for(nbh) + 2 * *tile_bits;
}

hipError_t task_order_temp_bytes(int64_t n, int key_bits, size_t* bytes) {
  *bytes = 0;
  if (n <= 1) return hipSuccess;
  return hipcub::DeviceRadixSort::SortPairs(nullptr, *bytes, static_cast<const uint64_t*>(nullptr),
                                            static_cast<uint64_t*>(nullptr), static_cast<const int32_t*>(nullptr),
                                            static_cast<int32_t*>(nullptr), (int)n, 0, key_bits, (hipStream_t)0);
}

hipError_t launch_task_order(const OrderArgs& a, hipStream_t s) {
  if (a.ntasks <= 1) return hipSuccess;
  hipLaunchKernelGGL(task_key_kernel, dim3((unsigned)((a.ntasks + 255) / 256)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  size_t bytes = a.temp_bytes;
  e = hipcub::DeviceRadixSort::SortPairs(a.temp, bytes, a.keys_in, a.keys_out, a.idx_in, a.order, (int)a.ntasks, 0,
                                         a.key_bits, s);
  if (e != hipSuccess || !a.tasks_out) return e;
  hipLaunchKernelGGL(task_gather_kernel, dim3((unsigned)((a.ntasks + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace bsa
