// Device-side validation of the metadata invariants the attention and
// transition kernels rely on (§3.1: the two blocks of a pair share one
// fidelity, and a BASE pair is two full blocks packed into one physical
// block; App. B.1: a transition starts from the opposite state).  Each
// check counts its violations and keeps the smallest index at which they
// occur.  Every read stays inside the arrays as their sizes declare them.
#include "ekv.h"
#include "common.h"
#include "launch.h"

namespace ekv {
namespace {

constexpr int kNone = 0x7fffffff;
constexpr int kThreads = 256;

__global__ void report_init_kernel(int32_t* report) {
  const int k = threadIdx.x;
  if (k < EKV_VIOL_COUNT) {
    report[k] = 0;
    report[EKV_VIOL_COUNT + k] = kNone;
  }
}

__device__ __forceinline__ void flag(int32_t* report, int kind, int index) {
  atomicAdd(report + kind, 1);
  atomicMin(report + EKV_VIOL_COUNT + kind, index);
}

// One thread per (sequence, logical block); the flat grid enumerates
// sequences times chunks of kThreads blocks.
__global__ __launch_bounds__(kThreads) void validate_batch_kernel(ValidateBatchArgs a) {
  const int chunks = (a.max_blocks + kThreads - 1) / kThreads;
  const int s = (int)(blockIdx.x / chunks);
  const int i = (int)(blockIdx.x % chunks) * kThreads + (int)threadIdx.x;
  if (s >= a.batch) return;
  const int row0 = s * a.max_blocks;   // host-checked: batch * max_blocks < 2^31

  const long long table_cap = (long long)a.max_blocks * kPage;
  const long long cap = a.max_seq_len > 0 ? min(table_cap, (long long)a.max_seq_len) : table_cap;
  const int raw = a.seq_lens[s];
  const bool structured = a.mode == EKV_MODE_STRUCTURED && a.bounds != nullptr;
  const int b0 = structured ? a.bounds[2 * s] : -1;
  const int b1 = structured ? a.bounds[2 * s + 1] : -1;
  if (i == 0) {
    if (raw < 0 || raw > cap) flag(a.report, EKV_VIOL_SEQ_LEN, row0);
    // a BASE pair range must be ordered; a negative start means "use the tags"
    if (structured && b0 >= 0 && b1 < b0) flag(a.report, EKV_VIOL_MODE, row0);
    if (structured && b0 < 0 && a.tags == nullptr) flag(a.report, EKV_VIOL_MODE, row0);
  }
  const int len = (int)max(0LL, min((long long)raw, table_cap));
  const int nblk = (len + kPage - 1) / kPage;
  if (i >= nblk) return;

  const int idx = row0 + i;
  const int e = a.bt[idx];
  if (e < 0 || e >= a.num_blocks) flag(a.report, EKV_VIOL_BLOCK_RANGE, idx);
  const int t = a.tags ? a.tags[idx] : 0;
  if (t > 1) flag(a.report, EKV_VIOL_TAG_VALUE, idx);
  if (i & 1) return;   // the pair checks run once, at member 0

  const int j = i >> 1;
  const bool has1 = i + 1 < nblk;
  const int e1 = has1 ? a.bt[idx + 1] : e;
  const int t1 = has1 && a.tags ? a.tags[idx + 1] : t;
  if (has1 && t != t1) flag(a.report, EKV_VIOL_PAIR_MIXED, idx);
  // the fidelity the attention kernels execute this pair at: the range in
  // structured mode, member 0's tag otherwise, nothing in native mode
  bool exec_base = false;
  if (a.mode == EKV_MODE_NATIVE) {
    if (t != 0 || t1 != 0) flag(a.report, EKV_VIOL_MODE, idx);
  } else if (structured && b0 >= 0) {
    exec_base = j >= b0 && j < b1;
    if (a.tags && (t != 0) != exec_base) flag(a.report, EKV_VIOL_MODE, idx);
  } else {
    exec_base = t != 0;
  }
  if (exec_base) {
    if (2LL * kPage * (j + 1) > len) flag(a.report, EKV_VIOL_BASE_PARTIAL, idx);
    else if (e1 != e) flag(a.report, EKV_VIOL_BASE_ALIAS, idx);
  }
}

// One thread per list entry.
__global__ __launch_bounds__(kThreads) void validate_list_kernel(ValidateListArgs a) {
  const int i = (int)(blockIdx.x * kThreads + threadIdx.x);
  if (i >= a.n) return;
  const int s = a.pairs[2 * i], j = a.pairs[2 * i + 1];
  for (int k = 0; k < i; ++k)
    if (a.pairs[2 * k] == s && a.pairs[2 * k + 1] == j) {
      flag(a.report, EKV_VIOL_LIST_DUPLICATE, i);
      break;
    }
  if (a.new_blocks) {
    const int b = a.new_blocks[i];
    if (b < 0 || b >= a.num_blocks) {
      flag(a.report, EKV_VIOL_NEW_BLOCK, i);
    } else {
      for (int k = 0; k < i; ++k)
        if (a.new_blocks[k] == b) {
          flag(a.report, EKV_VIOL_NEW_BLOCK, i);
          break;
        }
    }
  }
  if (s < 0 || s >= a.batch || j < 0 || 2LL * j + 1 >= a.max_blocks) {
    flag(a.report, EKV_VIOL_LIST_RANGE, i);
    return;
  }
  const size_t row = (size_t)s * a.max_blocks + 2 * j;
  const int e0 = a.bt[row], e1 = a.bt[row + 1];
  if (e0 < 0 || e0 >= a.num_blocks || e1 < 0 || e1 >= a.num_blocks) flag(a.report, EKV_VIOL_LIST_RANGE, i);
  const int want = a.kind == 0 ? EKV_TAG_TARGET : EKV_TAG_BASE;
  if (a.tags[row] != want || a.tags[row + 1] != want) flag(a.report, EKV_VIOL_LIST_STATE, i);
  if (a.seq_lens && 2LL * kPage * (j + 1) > a.seq_lens[s]) flag(a.report, EKV_VIOL_LIST_PARTIAL, i);
}

// Refinement: a visible table entry that holds one of the new blocks (one
// thread per (sequence, logical block), as the batch check).
__global__ __launch_bounds__(kThreads) void validate_in_use_kernel(ValidateListArgs a) {
  const int chunks = (a.max_blocks + kThreads - 1) / kThreads;
  const int s = (int)(blockIdx.x / chunks);
  const int i = (int)(blockIdx.x % chunks) * kThreads + (int)threadIdx.x;
  if (s >= a.batch) return;
  const int len = (int)max(0LL, min((long long)a.seq_lens[s], (long long)a.max_blocks * kPage));
  if (i >= (len + kPage - 1) / kPage) return;
  const int e = a.bt[(size_t)s * a.max_blocks + i];
  for (int k = 0; k < a.n; ++k)
    if (a.new_blocks[k] == e) {
      flag(a.report, EKV_VIOL_NEW_BLOCK, k);
      break;
    }
}

}  // namespace

hipError_t launch_validate_batch(const ValidateBatchArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(report_init_kernel, dim3(1), dim3(64), 0, st, a.report);
  if (a.batch > 0) {
    const long long grid = (long long)a.batch * ((a.max_blocks + kThreads - 1) / kThreads);
    hipLaunchKernelGGL(validate_batch_kernel, dim3((unsigned)grid), dim3(kThreads), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_validate_list(const ValidateListArgs& a, hipStream_t st) {
  hipLaunchKernelGGL(report_init_kernel, dim3(1), dim3(64), 0, st, a.report);
  if (a.n > 0) {
    hipLaunchKernelGGL(validate_list_kernel, dim3((a.n + kThreads - 1) / kThreads), dim3(kThreads), 0, st, a);
    if (a.kind == 1 && a.new_blocks && a.seq_lens && a.batch > 0) {
      const long long grid = (long long)a.batch * ((a.max_blocks + kThreads - 1) / kThreads);
      hipLaunchKernelGGL(validate_in_use_kernel, dim3((unsigned)grid), dim3(kThreads), 0, st, a);
    }
  }
  return hipGetLastError();
}

}  // namespace ekv
