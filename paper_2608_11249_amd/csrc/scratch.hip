// The library's static device scratch for callers that cannot allocate device
// memory (code under HIP graph capture, serving loops, harnesses that forbid
// hipMalloc): dlmc_entropy_cdf_noalloc keeps its CDF row tables and segment
// partials here instead of in buffers allocated per call.
//
// `scratch` is a file-scope device array; every GPU the library runs on holds
// its own copy until the process ends.  Host code never passes the array's
// name to a kernel (in host code it is only a stand-in symbol): the device
// address of each GPU's copy is looked up once per device with
// hipGetSymbolAddress, with that device current, and used from then on.
#include <mutex>

#include "kernels.h"

namespace dlmc {

// external linkage, so the runtime registers it under a stable name
__device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_lock;
void* g_addr[MAX_DEVICES] = {};

// slot i of a CDF launch with one "chunk" per row: row i, one committed row
__global__ void row_slots_kernel(int32_t* __restrict__ sel_row, int32_t* __restrict__ n_sel, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    sel_row[i] = i;
    n_sel[i] = 1;
  }
}

}  // namespace

void* scratch_address(int device) {
  DLMC_CHECK(device >= 0 && device < MAX_DEVICES, DLMC_E_INVAL, "device index out of range");
  std::lock_guard<std::mutex> g(g_lock);
  if (!g_addr[device]) {
    int cur = -1;
    DLMC_HIP(hipGetDevice(&cur));
    DLMC_CHECK(cur == device, DLMC_E_INVAL, "scratch lookup needs its device current");
    void* p = nullptr;
    DLMC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DLMC_CHECK(p != nullptr, DLMC_E_DEVICE, "no device address for the scratch array");
    g_addr[device] = p;
  }
  return g_addr[device];
}

void fill_row_slots(hipStream_t st, int32_t* sel_row, int32_t* n_sel, int n) {
  if (n <= 0) return;
  row_slots_kernel<<<ceil_div(n, 256), 256, 0, st>>>(sel_row, n_sel, n);
  DLMC_HIP(hipGetLastError());
}

}  // namespace dlmc
