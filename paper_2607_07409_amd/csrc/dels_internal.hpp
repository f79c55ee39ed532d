// Internal interface between the C ABI (api.cpp) and the kernel launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/dels.h"
#include "dels_device.hpp"

namespace dls {

// Turn the merged statistics of a whole row into the decoded token and row statistics.
// long_only marks a row decoded from the long logits alone.  A sampled row (temperature T)
// folded l / T into the fused log-sum-exp and l / T + g into the top-2: g_tok is the noise
// of the chosen token, so P.t1 - g_tok is l_tok / T.  Greedy rows pass g_tok = 0, temp = 1.
__device__ __forceinline__ void finalize_row(const Partial& P, float wl, float al, bool long_only,
                                             int32_t* tok, dls_row_stats* st, float* norm, float g_tok = 0.f,
                                             float temp = 1.f) {
  const int t = P.i1 == 0x7fffffff ? 0 : P.i1;   // every value -inf: the first index
  *tok = t;
  const float lse_l = lse_value(P.L);
  const float lse_s = long_only ? __builtin_nanf("") : lse_value(P.S);
  const float nr = long_only ? weighted(wl, lse_l) : __builtin_fmaf(al, lse_s, weighted(wl, lse_l));
  if (st) {
    const float ft = P.t1 - g_tok;   // l_tok / T
    st->score = ft * temp - nr;
    st->logprob = ft - lse_value(P.F);
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
bool combine_wide(int64_t rows, int32_t V);   // one 1024-thread workgroup per row
hipError_t launch_combine(const CombineArgs& a, hipStream_t st);

// adaptive fusion: the measure and gate of dls_adaptive in the form the kernels use
struct UncRule {
  int measure;           // DLS_UNC_ENTROPY or DLS_UNC_MAXPROB
  float inv_log_v;       // 1 / log V (0 when V = 1)
  float maxprob_scale;   // V / (V - 1) (0 when V = 1)
  float h_lo, inv_width; // g = clamp((u - h_lo) * inv_width, 0, 1)
};
struct UncArgs {
  const void* long_logits;
  dls_dtype dtype;
  int64_t rows;
  int32_t V;
  UncRule rule;
  float4* partials;          // rows * uncertainty_parts(rows, V) when that exceeds 1
  dls_row_uncertainty* out;  // rows
};
int uncertainty_parts(int64_t rows, int32_t V);
size_t uncertainty_workspace_bytes(int64_t rows, int32_t V);
hipError_t launch_uncertainty(const UncArgs& a, hipStream_t st);

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
  const float* alphas;       // [B] host per-position weights, or NULL (f.alpha everywhere)
  const float* betas;        // [B] host, or NULL (f.beta)
  Sampler smp;               // temperature sampling (smp.inv_temp = 0: greedy)
  const dls_row_uncertainty* unc;   // [batch, B] adaptive-fusion gates, or NULL (gate 1)
};
hipError_t launch_draft(const DraftArgs& a, hipStream_t st);

hipError_t launch_accept(const int32_t* draft, const int32_t* target, int32_t batch, int32_t B,
                         int32_t* out, hipStream_t st);
hipError_t launch_unigram_prior(const int32_t* tokens, int64_t n, int32_t V, float smoothing, uint64_t* counts,
                                float* out, hipStream_t st);

// ------------------------------------------------------------------------------------------
// prepared heads and the persistent drafting kernel
// ------------------------------------------------------------------------------------------
constexpr int kMaxBatch = 64;              // sequences per call on the persistent path
constexpr int kMaxG = 256;                 // workgroups (one per CU of a gfx950)
constexpr size_t kMaxLds = 160 * 1024;     // LDS per CU on gfx950
constexpr int kNarrowBatch = 4;            // the persistent kernel's narrow form: at most 4 sequences
constexpr int kMaxH = 16 * kMaxG;          // GRU hidden units on the persistent path (16 per GRU workgroup)
constexpr size_t kH32Set = (size_t)2 * kMaxBatch * kMaxH;   // words of one set of the wide h hand-off
constexpr uint64_t kPreparedMagic = 0x50455250534c4544ull;

struct PreparedHeader {
  uint64_t magic;
  int32_t V, d, H, r;
  const void *emb, *w_ih, *w_hh, *w_vocab;
};
struct PreparedLayout {
  int NT, KK;
  size_t off_T, off_wv, off_whh, total;
};
PreparedLayout prepared_layout(const dls_local_head& h);
hipError_t launch_prepare(const dls_local_head& h, void* buf, hipStream_t st);

// error word of a persistent drafting workspace (the second uint32 of its header)
constexpr uint32_t kErrStalled = DLS_DRAFT_ERR_STALLED;
constexpr uint32_t kErrPrepared = DLS_DRAFT_ERR_PREPARED;
hipError_t launch_copy_word(const uint32_t* src, int32_t* dst, hipStream_t st);

// the scratch of dls_draft_block_noalloc (noalloc.hip): the device address of the current
// device's copy, and the check that restores it after a failed call
constexpr size_t kNoallocScratchBytes = DLS_NOALLOC_SCRATCH_BYTES;
void* noalloc_scratch(int dev, hipError_t* err);
hipError_t launch_scratch_guard(void* dev_scratch, hipStream_t st);

struct PersistArgs {
  const PreparedHeader* prep;   // header of the prepared buffer, and what it must hold
  PreparedHeader expect;
  const float* T;            // folded input projection [V][3H]
  const uint4* wv;           // W_vocab tiles in MFMA operand order
  const uint4* whh;          // W_hh in MFMA operand order, per 16-unit group
  const bf16_t* w_rank;      // [r][H]
  const bf16_t* e_m;         // Markov head: E_M [V][r] (the GRU fields are unused then)
  int V, H, r, NT, NG, rpg, cap_a, gcap, rows_max;
  size_t lds_region_a;
  const void* L;             // long logits [batch][B][V]
  const int32_t* last;
  const float* prior;
  int batch, B;
  float wl;
  float al_j[64], be_j[64];  // fusion weights of each draft position (B <= 64)
  int literal;
  Sampler smp;               // temperature sampling (smp.inv_temp = 0: greedy)
  const dls_row_uncertainty* unc;   // [batch, B] adaptive-fusion gates, or NULL (gate 1)
  int ordinary_launch;       // host only: ordinary instead of cooperative dispatch
  int32_t* out_tokens;
  dls_row_stats* out_stats;
  uint32_t* hdr;             // [0] call epoch, [1] error word
  uint64_t* keys;            // [2 sets][2 parities][kMaxBatch][G]
  uint64_t* hbuf;            // [2 parities][batch][H] (narrow batches)
  uint32_t* h32;             // wide batches' h: [2 sets][2 parities][hrep][batch][H] in a set stride of
                             // kH32Set words; 24-bit h | 8-bit position tag; cleared by every call
  int hrep;                  // replicas of the wide h words (a power of two, 2 hrep batch H <= kH32Set)
  uint64_t* rbuf;            // [replicas][2 parities][batch][r]
  uint64_t* stats;           // [B][batch][G][8] tagged LSE partials
  uint64_t* tokw;            // merged tokens of wide batches: [2 parities][kMaxBatch] tagged words
};
struct PersistPlan {
  bool ok;
  const char* why;
  int G, NG, rpg, NT, cap_a, gcap, rows_max;
  size_t lds_region_a, lds;
};
struct PersistWorkspace {
  size_t off_keys, off_h, off_h32, off_rho, off_tokw, off_stats, total;
};
__host__ __device__ inline void persist_tile_range(int w, int G, int NG, int NT, int cap_a, int gcap, int* t0,
                                                   int* n);
PersistPlan persist_plan(const dls_local_head& h, int32_t batch, int32_t B, dls_dtype long_dtype, bool prior, int G);
PersistWorkspace persist_workspace(const dls_local_head& h, int32_t batch, int32_t B);
hipError_t launch_persistent(const PersistArgs& pa, const PersistPlan& pl, dls_dtype long_dtype, hipStream_t st);

}  // namespace dls
