// Energy and forces without device allocation: compute_energy_forces_noalloc.
//
// Some callers cannot allocate device memory while they run: code under HIP
// graph capture, tight serving loops, harnesses that forbid it.  For them the
// per-call buffers of an evaluation (compaction maps, edge records, reverse
// index, node state and its gradient, energy partials, folded species index)
// live in one file-scope device array of kNoAllocScratchBytes instead of the
// model's grow-only workspace.  Each device holds its own copy of the array
// until the process ends.  Its device address is looked up once per device,
// when the first model is created there, and only that address reaches the
// kernels.
//
// Every call on a device shares that device's array and leaves the last
// call's contents in it; nothing in it needs to start at zero (the only
// counter is cleared by a fill kernel at the start of each call).  Calls
// that overlap on one device race on the array.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/dpa4c.h"
#include "launch.h"

namespace dpa4c {

namespace {

constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::mutex g_scratch_lock;
void* g_scratch_ptr[kMaxDevices] = {};

void* scratch_of(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_lock);
  return g_scratch_ptr[device];
}

}  // namespace

int noalloc_setup(int device) {
  if (device < 0 || device >= kMaxDevices) {
    set_error("the no-allocation entry point supports device indices below 64");
    return DPA4C_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_scratch_lock);
  if (g_scratch_ptr[device]) return 0;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) {
    set_error(std::string("hipGetSymbolAddress of the no-allocation scratch: ") +
              hipGetErrorString(e));
    return DPA4C_ERR_HIP;
  }
  g_scratch_ptr[device] = p;
  return 0;
}

}  // namespace dpa4c

using namespace dpa4c;

extern "C" int compute_energy_forces_noalloc(const dpa4c_model* m, const double* pos,
                                             const int32_t* species, int64_t N,
                                             const double cell[9], const int pbc[3], double r_c,
                                             const int64_t* row_ptr, const int32_t* nbr_j,
                                             const int32_t* nbr_shift, int64_t n_pairs,
                                             double* e_atom, double* forces, double* e_total,
                                             void* stream) {
  if (!m || N < 0 || n_pairs < 0) {
    set_error("compute_energy_forces_noalloc: bad pointer or size");
    return DPA4C_ERR_INVALID_ARG;
  }
  unsigned char* base = static_cast<unsigned char*>(scratch_of(m->device));
  if (!base) {
    set_error("compute_energy_forces_noalloc: no scratch on the model's device");
    return DPA4C_ERR_INVALID_ARG;
  }
  size_t sizes[kEvalBufs];
  eval_buf_sizes(N, n_pairs, m->S + 2, sizes);
  size_t total = 0;
  for (size_t b : sizes) total += b;
  if (total > kNoAllocScratchBytes) {
    set_error("compute_energy_forces_noalloc: " + std::to_string(N) + " atoms and " +
              std::to_string(n_pairs) + " list entries need " + std::to_string(total) +
              " bytes of scratch, more than its " + std::to_string(kNoAllocScratchBytes) +
              " bytes");
    return DPA4C_ERR_INVALID_ARG;
  }
  unsigned char* at = base;
  auto take = [&](int k) {
    unsigned char* p = at;
    at += sizes[k];
    return p;
  };
  EvalBufs b{};
  b.ecount = reinterpret_cast<int32_t*>(take(0));
  b.edge = reinterpret_cast<float4*>(take(1));
  b.cskin = reinterpret_cast<int32_t*>(take(2));
  b.skin_rev = reinterpret_cast<int64_t*>(take(3));
  b.node = reinterpret_cast<float*>(take(4));
  b.node_grad = reinterpret_cast<float*>(take(5));
  b.epart = reinterpret_cast<double*>(take(6));
  b.fidx = reinterpret_cast<int32_t*>(take(7));
  b.fold_mask = reinterpret_cast<uint32_t*>(take(8));
  b.check = reinterpret_cast<int64_t*>(take(9));
  return energy_forces_core(m, pos, species, N, cell, pbc, r_c, row_ptr, nbr_j, nbr_shift, n_pairs,
                            e_atom, forces, e_total, nullptr, nullptr, &b, stream);
}
