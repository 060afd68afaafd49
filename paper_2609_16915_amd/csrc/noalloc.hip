// Allocation-free variant of the PBS entry point, for callers that cannot
// allocate device memory while they run (code under HIP graph capture,
// tight serving loops, harnesses that forbid hipMalloc).
//
// The only scratch of a PBS is the buffer of extracted ciphertexts
// [batch][N+1] between the blind-rotation and key-switching kernels.  Here
// it is a file-scope static device array of ROSETTA_NOALLOC_SCRATCH_BYTES,
// which every GPU the library runs on holds until the process ends.  Host
// code never passes the array's name to a kernel (on the host it is only a
// stand-in for the symbol): on the first call on a device, with that device
// current, hipGetSymbolAddress gives this device's address of its copy, and
// that address is what the kernels receive.
//
// Every call on one device shares that device's array.  Calls on one stream
// run in order and are safe; calls that overlap in time on one device (two
// streams, two threads) race on it.  Nothing needs clearing between calls:
// the blind-rotation kernel writes every word of the batch's extracted
// ciphertexts before the key switch reads them.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "internal.hpp"
#include "rosetta.h"

static __device__ __align__(256) uint64_t scratch[ROSETTA_NOALLOC_SCRATCH_BYTES / 8];

namespace {

std::mutex g_scratch_mu;
std::map<int, uint64_t *> g_scratch_ptr;  // device -> its copy of `scratch`

}  // namespace

extern "C" rosetta_status rosetta_pbs_batch_noalloc(const uint64_t *lwe_in,
                                                    const uint64_t *bsk_dev,
                                                    const uint64_t *ksk_dev, const uint64_t *lut,
                                                    uint64_t *lwe_out, size_t batch,
                                                    const rosetta_params *params, void *stream) {
  rosetta_status st = rosetta_check_params(params);
  if (st) return st;
  if (batch == 0) return ROSETTA_OK;
  if (!lwe_in || !bsk_dev || !ksk_dev || !lut || !lwe_out) {
    rosetta::set_last_error("NULL pointer argument");
    return ROSETTA_ERR_NULL;
  }
  const size_t need = rosetta_pbs_workspace_bytes(params, batch);
  if (need > ROSETTA_NOALLOC_SCRATCH_BYTES) {
    char msg[256];
    snprintf(msg, sizeof msg,
             "batch %zu at N = %u needs %zu bytes of scratch; the static scratch holds %zu "
             "(at most %zu ciphertexts at this N)",
             batch, params->N, need, (size_t)ROSETTA_NOALLOC_SCRATCH_BYTES,
             (size_t)ROSETTA_NOALLOC_SCRATCH_BYTES / (((size_t)params->N + 1) * 8));
    rosetta::set_last_error(msg);
    return ROSETTA_ERR_SIZE;
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    rosetta::set_last_error(hipGetErrorString(e));
    return ROSETTA_ERR_DEVICE;
  }
  uint64_t *ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch_ptr.find(dev);
    if (it == g_scratch_ptr.end()) {
      e = hipGetSymbolAddress((void **)&ptr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !ptr) {
        char msg[256];
        snprintf(msg, sizeof msg, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                 hipGetErrorString(e));
        rosetta::set_last_error(msg);
        return ROSETTA_ERR_DEVICE;
      }
      it = g_scratch_ptr.emplace(dev, ptr).first;
    }
    ptr = it->second;
  }
  // the two kernels of rosetta_pbs_batch_ws, with this device's scratch as
  // the workspace (the twiddle tables live in static device memory too)
  return rosetta_pbs_batch_ws(lwe_in, bsk_dev, ksk_dev, lut, lwe_out, batch, params, ptr,
                              ROSETTA_NOALLOC_SCRATCH_BYTES, stream);
}
