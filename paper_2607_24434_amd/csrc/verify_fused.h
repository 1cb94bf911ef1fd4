// The verify layer in one launch: argument block and launcher
// (internal).
#pragma once

#include "de_common.h"

namespace de {

struct FusedArgs {
  // The gate/up half: the block of positions x, the fused selection and union
  // (sel, fuse_route and fuse_select set), the routed source with its tagged
  // A_r (a_tag) and the shared block as dense[0] with its tagged A_s (out_tag).
  GroupedArgs gu;
  // The down half: the same routed source with its tagged P_r (p_tag; the
  // plain P_r is written too) and the shared down projection in column chunks
  // (dense[0..n_dense), each reading its tagged input through vin_tag and
  // writing a tagged [T, H] partial through out_tag).
  GroupedArgs dn;
  // y, normed, residual, eps, T, H, kk (top-k), n_dense: the combine of the
  // separate launches, with the partials read from the tagged buffers.
  CombineArgs c;
  int region_floats;   // LDS floats of the staged rows (positions, or a down source's inputs)
  int32_t* status;     // device status word
  uint64_t* pub;       // the published lists (verify_fused_pub_words tagged words)
  // Set by the launcher: gate/up blocks, down blocks, down runs per source
  // and tiles per run.
  int g1, g2, runs, run_tiles;
};

// LDS bytes of a block for the shape (0 when the shape does not fit the
// kernel): T positions of H, top-k of N, routed intermediate I, shared
// intermediate Is split into `chunks` down chunks.
size_t verify_fused_lds(int T, int H, int N, int k, int I, int Is, int chunks);
// Floats of the staged-rows region for the shape.
int verify_fused_region(int T, int H, int I, int Is, int chunks);
// Tagged words of the published lists.
size_t verify_fused_pub_words(int T, int N, int k);
// One launch of gate/up, down and combine blocks (two 512-thread blocks per
// CU resident).
hipError_t launch_verify_fused(const FusedArgs& f, size_t lds, hipStream_t s);

// Host side (api.cpp): true only when DE_VERIFY_FUSED is "1".
bool verify_fused_enabled();

}  // namespace de
