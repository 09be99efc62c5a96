// uattn_decode_noalloc: the token-wise decode with its workspace taken from a
// library-owned static device array instead of the caller's buffer, for
// callers that cannot allocate device memory (code under HIP graph capture,
// serving loops that forbid allocation).
//
// `scratch` below is a file-scope device array.  Its name, used in host
// code, is a host-side stand-in and not a device address, so host code never
// passes it anywhere: on each device, the first call looks up the array's
// device address with hipGetSymbolAddress (with that device current) and
// keeps it; every kernel argument and size below is derived from that
// address.  Each device holds its own copy of the array until the process
// ends.
//
// Every call zeroes the arrival counters at the array's start with a fill
// kernel (a kernel, not a memset node, so that the call can be captured and
// replayed), then runs the same decode kernel as uattn_decode with the array
// as its workspace.  All calls on one device share the array: calls that
// overlap on a device (different streams, no ordering) race on it.
#include <mutex>

#include "uattn_internal.h"

namespace {

constexpr size_t kScratchBytes = UATTN_DECODE_SCRATCH_BYTES;

__device__ __attribute__((aligned(256))) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void* g_scratch_ptr[kMaxDevices] = {nullptr};

// Device address of this device's copy of `scratch` (nullptr on failure).
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

__global__ __launch_bounds__(256) void zero_words(uint4* p, int n16) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n16) p[i] = uint4{0u, 0u, 0u, 0u};
}

}  // namespace

extern "C" {

size_t uattn_decode_scratch_limit(void) { return kScratchBytes; }

uattn_status uattn_decode_noalloc(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                                  const int32_t* seqlens, int32_t batch, int32_t max_pages_per_seq, int32_t page_size,
                                  int32_t num_pages, int32_t max_seqlen, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, float softmax_scale, void* out, float* lse, void* stream) {
  // host arithmetic only: sizes beyond the array are refused before any HIP call
  const size_t need = uattn_decode_workspace_bytes(batch, max_seqlen, num_q_heads, head_dim);
  if (need > kScratchBytes) return UATTN_ESCRATCH;
  void* ws = nullptr;
  if (need > 0 && batch > 0) {
    ws = scratch_address();
    if (ws == nullptr) return UATTN_ELAUNCH;
  }
  uattn::DecodeLaunch a;
  const uattn_status st =
      uattn::decode_prepare(q, k_pages, v_pages, block_table, seqlens, batch, max_pages_per_seq, page_size, num_pages,
                            max_seqlen, num_q_heads, num_kv_heads, head_dim, softmax_scale, out, lse, ws,
                            ws != nullptr ? kScratchBytes : 0, &a);
  if (st != UATTN_OK || a.batch == 0) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (a.ws_cnt != nullptr) {
    // the counter region the decode relies on being zero (a multiple of 256 bytes)
    const int n16 = static_cast<int>(uattn::decode_ws_cnt_bytes(batch, num_q_heads) / 16);
    hipLaunchKernelGGL(zero_words, dim3((n16 + 255) / 256), dim3(256), 0, s, static_cast<uint4*>(ws), n16);
    if (hipGetLastError() != hipSuccess) return UATTN_ELAUNCH;
  }
  return uattn::launch_decode(a, s) == hipSuccess ? UATTN_OK : UATTN_ELAUNCH;
}

}  // extern "C"
