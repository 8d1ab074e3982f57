// Skip-gram pairs without a caller workspace, for callers that cannot allocate
// device memory (code under stream capture, tight serving loops, harnesses that
// forbid hipMalloc).
//
// rdf2v_skipgram_pairs takes its scratch (per-walk output offsets and the scan's
// block sums) from a caller workspace. This variant keeps that scratch in one
// fixed file-scope device array instead. HIP gives every device that loads
// this code object its own copy of the array, at its own address; the host
// name `scratch` is only a stand-in for it, so the device address is looked up
// once per device with hipGetSymbolAddress and only that address is ever
// handed to kernels. The kernels are those of rdf2v_skipgram_pairs.
//
// Every call on one device uses the same array: calls that overlap in time on
// one device (different streams, or threads) race on it. Nothing in it has to
// start at zero: within a call every word is written before it is read.

#include <mutex>

#include "common.hpp"
#include "launch.hpp"

namespace rdf2v {
namespace {

static_assert(RDF2V_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size must keep 256-byte alignment");

// The library-held scratch of rdf2v_skipgram_pairs_noalloc (one copy per device).
static __device__ __align__(256) unsigned char scratch[RDF2V_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 256;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch` on each device, once looked up

// Device address of `scratch` on `device`, looked up on the first call for that
// device with the device made current for the lookup (and the caller's current
// device restored afterwards).
rdf2v_status scratch_address(int device, void **out) {
  if (device < 0 || device >= kMaxDevices) return RDF2V_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[device] == nullptr) {
    int current = -1;
    RDF2V_HIP_TRY(hipGetDevice(&current));
    if (current != device) RDF2V_HIP_TRY(hipSetDevice(device));
    void *ptr = nullptr;
    const hipError_t err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (current != device) RDF2V_HIP_TRY(hipSetDevice(current));
    if (err != hipSuccess || ptr == nullptr) return RDF2V_ERR_HIP;
    g_scratch_ptr[device] = ptr;
  }
  *out = g_scratch_ptr[device];
  return RDF2V_OK;
}

}  // namespace
}  // namespace rdf2v

RDF2V_API rdf2v_status rdf2v_skipgram_pairs_noalloc(const int32_t *tokens, const int32_t *len, int64_t num_walks,
                                                    int32_t row_width, int32_t window, int32_t *pairs_out,
                                                    int64_t pair_capacity, int64_t *pair_count_out,
                                                    int32_t *status_dev, void *stream) {
  if (num_walks < 0 || window < 0 || pair_capacity < 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (row_width < 1 || row_width > 2 * RDF2V_MAX_DEPTH + 1) return RDF2V_ERR_INVALID_ARGUMENT;
  if (pair_count_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > 0 && (tokens == nullptr || len == nullptr)) return RDF2V_ERR_INVALID_ARGUMENT;
  if (pair_capacity > 0 && pairs_out == nullptr) return RDF2V_ERR_INVALID_ARGUMENT;
  if ((reinterpret_cast<uintptr_t>(pairs_out) & 7) != 0) return RDF2V_ERR_INVALID_ARGUMENT;
  if (num_walks > RDF2V_NOALLOC_MAX_WALKS) return RDF2V_ERR_TOO_LARGE;
  if (rdf2v::skipgram_workspace_bytes(num_walks) > size_t(RDF2V_NOALLOC_SCRATCH_BYTES)) return RDF2V_ERR_TOO_LARGE;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  int device = -1;
  if (s == nullptr)
    RDF2V_HIP_TRY(hipGetDevice(&device));  // the null stream belongs to the current device
  else
    RDF2V_HIP_TRY(hipStreamGetDevice(s, &device));
  void *ws = nullptr;
  const rdf2v_status st = rdf2v::scratch_address(device, &ws);
  if (st != RDF2V_OK) return st;
  return rdf2v::launch_skipgram_pairs(tokens, len, num_walks, row_width, window, pairs_out, pair_capacity,
                                      pair_count_out, ws, status_dev, s);
}
