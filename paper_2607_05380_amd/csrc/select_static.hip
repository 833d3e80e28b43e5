// pack_select_static(): the greedy selection of pack_select() with its scratch
// in a file-scope device array instead of a caller's workspace, for callers
// that cannot allocate device memory.
//
// The array `scratch` (kSelectStaticBytes, 256-byte aligned) exists once per
// GPU the library runs on and lives until the process ends.  In host code its
// name is only a host-side stand-in, so its device address is taken with
// hipGetSymbolAddress on the first call on each device (with that device
// current) and kept per device; that address, never the name, is what the
// kernels receive.  Every call on one GPU shares that GPU's array: the
// selection's own first kernel initialises every value it later reads, and
// calls that overlap on one GPU (concurrent streams or threads) race.
#include <mutex>

#include "../../include/tabpack.h"
#include "pack_internal.h"

namespace {

constexpr size_t kSelectStaticBytes = PACK_SELECT_STATIC_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kSelectStaticBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// The device address of this device's copy of `scratch` (nullptr on failure,
// with the library's last error set).
void* scratch_ptr(int* rc) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    *rc = tabpack::set_error(PACK_EHIP, hipGetErrorString(e));
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    *rc = tabpack::set_error(PACK_EINVAL, "device ordinal beyond the static scratch table");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      *rc = tabpack::set_error(PACK_EHIP, e != hipSuccess ? hipGetErrorString(e) : "no address for the scratch array");
      return nullptr;
    }
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

int pack_select_static(pack_handle* h, const float* cand, const void* yv, int32_t C, int64_t Nv, int32_t m_ens,
                       int32_t* sel_out, int32_t* n_sel_out, double* score_out, hipStream_t stream) {
  if (!h) return tabpack::set_error(PACK_EINVAL, "handle is NULL");
  size_t need = 0;
  const int rc0 = pack_select_workspace_size(C, Nv, &need);
  if (rc0 != PACK_OK) return rc0;
  if (need > kSelectStaticBytes)
    return tabpack::set_error(PACK_EINVAL, "pack_select_static: C and Nv need more scratch than the "
                                           "PACK_SELECT_STATIC_BYTES of the static array; use pack_select with a "
                                           "workspace");
  int rc = PACK_OK;
  void* p = scratch_ptr(&rc);
  if (!p) return rc;
  return tabpack::select_with_scratch(h, cand, yv, C, Nv, m_ens, p, kSelectStaticBytes, sel_out, n_sel_out,
                                      score_out, stream);
}
