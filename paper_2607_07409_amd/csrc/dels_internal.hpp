// Internal interface between the C ABI (api.cpp) and the kernel launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/dels.h"
#include "dels_device.hpp"

namespace dls {

// Turn the merged statistics of a whole row into the decoded token and row statistics.
// has_short = false marks a row decoded from the long logits alone.
__device__ __forceinline__ void finalize_row(const Partial& P, float wl, float al, bool long_only,
                                             int32_t* tok, dls_row_stats* st, float* norm) {
  const int t = P.i1 == 0x7fffffff ? 0 : P.i1;   // every value -inf: the first index
  *tok = t;
  const float lse_l = lse_value(P.L);
  const float lse_s = long_only ? __builtin_nanf("") : lse_value(P.S);
  const float nr = long_only ? wl * lse_l : __builtin_fmaf(al, lse_s, wl * lse_l);
  if (st) {
    st->score = P.t1 - nr;
    st->logprob = P.t1 - lse_value(P.F);
    st->gap = P.t1 - P.t2;
    st->lse_long = lse_l;
    st->lse_short = lse_s;
    st->lse_fused = lse_value(P.F);
  }
  if (norm) *norm = nr;
}

struct CombineArgs {
  const void* long_logits;
  const void* short_logits;
  dls_dtype dtype;
  const float* prior;
  int64_t rows;
  int32_t V;
  float wl, al, be;
  int parts;
  Partial* partials;   // rows * parts (parts > 1)
  float* norm;         // rows
  int32_t* out_token;
  dls_row_stats* out_stats;
  float* out_scores;
};
int combine_parts(int64_t rows, int32_t V);
hipError_t launch_combine(const CombineArgs& a, hipStream_t st);

struct DraftLayout {
  int slice;       // vocabulary rows per workgroup of the LM-head phase
  int groups;      // number of such workgroups
  size_t off_h0, off_h1, off_rho, off_tok, off_part, total;
};
DraftLayout draft_layout(const dls_local_head& h, int32_t batch, int32_t B);

struct DraftArgs {
  dls_local_head head;
  const void* long_logits;
  dls_dtype long_dtype;
  const int32_t* last_token;
  const float* prior;
  int32_t batch, B;
  dls_fusion f;
  int32_t* out_tokens;
  dls_row_stats* out_stats;
  char* ws;
  DraftLayout lay;
};
hipError_t launch_draft(const DraftArgs& a, hipStream_t st);

hipError_t launch_accept(const int32_t* draft, const int32_t* target, int32_t batch, int32_t B,
                         int32_t* out, hipStream_t st);

}  // namespace dls
