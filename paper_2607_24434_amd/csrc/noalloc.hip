// de_verify_layer for callers that cannot allocate device memory (code under
// HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
// the layer's scratch is a file-scope device array instead of a caller
// workspace.  Every call on one GPU shares that GPU's copy of the array, so
// calls that overlap on one GPU race.
#include "../../include/draftexpert.h"
#include "de_common.h"

#include <mutex>

namespace de {
int verify_layer_chain(const de_moe_desc* d, int T, const float* x, const float* w_router,
                       const float* bias, const de_expert_table* routed, const void* shared_w,
                       float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                       int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                       int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                       hipStream_t stream, bool logits_ready, const float* next_router);
}  // namespace de

namespace {

// Largest layer scratch this entry point serves (de_workspace_bytes of the
// call's shape and block length): the V2-Lite layer up to T = 64 needs about
// 8.5 MB.
constexpr size_t kScratchBytes = 16u << 20;
constexpr size_t kCtlBytes = 4096;  // the layer scratch's control area (counters, status, flags)

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

__global__ void clear_words(uint32_t* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// The device address of this device's copy of `scratch`, resolved once per
// device (with that device current); its control area is zeroed on first use
// by a fill kernel on `stream`.  NULL on failure.
void* device_scratch(hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (de::note_hip(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess || p == nullptr)
      return nullptr;
    const int n = (int)(kCtlBytes / 4);
    hipLaunchKernelGGL(clear_words, dim3((n + 255) / 256), dim3(256), 0, stream,
                       static_cast<uint32_t*>(p), n);
    if (de::note_hip(hipGetLastError()) != hipSuccess) return nullptr;
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" {

size_t de_noalloc_scratch_bytes(void) { return kScratchBytes; }

int de_verify_layer_noalloc(const de_moe_desc* d, int T, const float* x, const float* w_router,
                            const float* bias, const de_expert_table* routed, const void* shared_w,
                            float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                            int32_t* union_ids, int32_t* offsets, int32_t* tok_list,
                            float* gate_list, int32_t* pair_pos, const de_epilogue* epi,
                            hipStream_t stream) {
  const size_t need = de_workspace_bytes(d, T);
  if (need == 0) {
    const int rc = de_check_desc(d);
    return rc != DE_OK ? rc : DE_ERR_INVALID;
  }
  if (need > kScratchBytes) return DE_ERR_WORKSPACE;
  void* ws = device_scratch(stream);
  if (ws == nullptr) return DE_ERR_HIP;
  return de::verify_layer_chain(d, T, x, w_router, bias, routed, shared_w, y, topk_idx,
                                topk_gate, n_union, union_ids, offsets, tok_list, gate_list,
                                pair_pos, epi, ws, kScratchBytes, stream, false, nullptr);
}

}  // extern "C"
