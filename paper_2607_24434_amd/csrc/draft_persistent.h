// The persistent draft pass: argument block and launcher (internal).
#pragma once

#include "de_common.h"

namespace de {

constexpr int kPDMaxH = 2048;      // hidden size the kernel keeps in LDS
constexpr int kPDMaxLayers = 32;   // layers per launch (their descriptors ride in the kernel arguments)
constexpr int kPDMaxGrid = 256;    // blocks (one per CU)

// One MoE layer of the run (bf16 weights).
struct PDLayer {
  const float* w_router;          // [N, H] fp32
  const float* bias;              // [N] or NULL
  const char* routed;             // expert table base
  int64_t stride;                 // bytes per slot
  const int32_t* slot_of_expert;  // [N] or NULL (identity)
  const char* shared;             // shared block [G|U|D], intermediate Is
  const char* draft;              // draft block [G|U|D], intermediate Id (NULL when Id is 0)
  int32_t n_slots;
  float gamma;
};

struct PDShape {
  int H, N, k, I, Is, Id;
  int n_chunks, chunk;            // the shared down projection in n_chunks column chunks
};

struct PDArgs {
  int L;                          // layers in this launch
  int H, N, k, I, Is, Id;
  int n_chunks, chunk;
  int has_draft;                  // Id > 0 (every layer has a draft block)
  int score_func, norm_topk;
  float routed_scale, eps;
  int grid;                       // blocks (one per CU)
  unsigned spin_limit;            // polls before a wait gives up
  size_t lds_bytes;               // dynamic LDS per block
  const float* x_in;              // [H] the first layer's input RMSNorm(h)
  const float* h_in;              // [H] its residual, or NULL (y = layer(x))
  const float* z_in;              // [N] its router logits, or NULL (computed here)
  float* y_out;                   // [H] the last layer's y
  float* normed_out;              // [H] RMSNorm(y), or NULL
  int32_t* pred_idx;              // [L, k] the top-k of every layer, or NULL
  float* pred_gate;               // [L, k] their gates, or NULL
  float* a_buf;                   // [Is + Id + I] gate/up outputs
  // [H] per-row sums of the down partials as (value, tag) words, tagged like
  // the logit words.
  uint64_t* d_tag;
  // [N] router logits as 64-bit words (value, tag): the tag in the high half
  // is (epoch << 6) + layer + 1, so a word of another layer or launch is never
  // taken for this one's.
  uint64_t* z_tag;
  float* z_plain;                 // [N] the last selected layer's logits (the workspace's logit row)
  // Arrival flags, one 64-bit word per block: (epoch << 32) | arrivals so
  // far.  The epoch grows with every launch, so flags left by earlier
  // launches are always below this launch's values and nothing is reset.
  uint64_t* grid_flags;           // [grid]
  uint32_t epoch;
  int32_t* status;                // device status word
  PDLayer layers[kPDMaxLayers];
};

// True when the shape fits the kernel's static tiling for `grid` blocks;
// gu_it / dn_it receive the 16-byte iterations per lane of a gate/up row and of
// a down row.
bool draft_persistent_fits(const PDShape& s, int grid, int* gu_it, int* dn_it);
// Dynamic LDS of a block.
size_t draft_persistent_lds(const PDShape& s);
hipError_t launch_draft_persistent(const PDArgs& a, hipStream_t s);

// Host side (api.cpp).
constexpr int kPDNotApplicable = 1;
bool draft_persistent_enabled();

}  // namespace de
