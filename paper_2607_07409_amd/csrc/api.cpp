// C ABI of libdels: argument checks (host only, before any HIP call), workspace
// sizing, device checks and dispatch to the kernel launchers.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <type_traits>

#include "dels_internal.hpp"
#include "peaks.hpp"

namespace {

// Process-lifetime state of the library is trivially destructible (plain arrays and flags):
// the library registers no destructor that would run at process exit.
thread_local char g_last_error[512];

void clear_error() { g_last_error[0] = 0; }

dls_status fail(dls_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
dls_status fail(dls_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return s;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Device check: a visible gfx950 device must be current.  The result for each device
// id is computed once; it never changes during the life of the process.
struct DevInfo {
  std::once_flag once;
  bool ok;
  int cus;
  char why[160];
};
static_assert(std::is_trivially_destructible<DevInfo>::value, "no exit-time destructor");
DevInfo g_dev[64];

dls_status check_device(int* cus = nullptr) {
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n <= 0) return fail(DLS_ERR_DEVICE, "no HIP device available (%s)", hipGetErrorString(e));
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess)
    return fail(DLS_ERR_DEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= 64) return fail(DLS_ERR_DEVICE, "device id %d out of range", dev);
  DevInfo& di = g_dev[dev];
  std::call_once(di.once, [&]() {
    hipDeviceProp_t p;
    hipError_t pe = hipGetDeviceProperties(&p, dev);
    if (pe != hipSuccess) {
      snprintf(di.why, sizeof di.why, "hipGetDeviceProperties failed: %s", hipGetErrorString(pe));
      return;
    }
    if (std::strncmp(p.gcnArchName, "gfx950", 6) != 0) {
      snprintf(di.why, sizeof di.why, "device is %s, the library is built for gfx950 only", p.gcnArchName);
      return;
    }
    int coop = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, dev) != hipSuccess) coop = 0;
    di.cus = coop ? p.multiProcessorCount : 0;
    di.ok = true;
  });
  if (!di.ok) return fail(DLS_ERR_DEVICE, "%s", di.why);
  if (cus) *cus = di.cus;
  return DLS_OK;
}

// number of persistent workgroups for this device (0: no cooperative launch)
int persist_groups(int cus) { return std::min(cus, dls::kMaxG); }

dls_status hip_fail(hipError_t e, const char* what) {
  return fail(DLS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// An enum from a C caller may hold any int; loading an out-of-range value as the C++ enum is
// undefined, so caller-supplied enums are read through their representation until validated.
template <typename E>
int enum_bits(const E& e) {
  static_assert(sizeof(E) == sizeof(int), "the C enums of the ABI are int-sized");
  int v;
  std::memcpy(&v, &e, sizeof v);
  return v;
}

bool valid_dtype(int t) { return t == DLS_F32 || t == DLS_BF16; }

dls_status check_fusion(const dls_fusion& f) {
  if (!std::isfinite(f.w_long) || !std::isfinite(f.alpha) || !std::isfinite(f.beta))
    return fail(DLS_ERR_ARG, "fusion weights must be finite");
  if (f.flags & ~(DLS_FIRST_ROW_LONG_ONLY | DLS_EXCLUSIVE_DEVICE))
    return fail(DLS_ERR_ARG, "unknown fusion flags 0x%x", f.flags);
  return DLS_OK;
}

dls_status check_rule(const dls_adaptive& r) {
  if (r.measure != DLS_UNC_ENTROPY && r.measure != DLS_UNC_MAXPROB)
    return fail(DLS_ERR_ARG, "unknown uncertainty measure %d", r.measure);
  if (r.reserved != 0) return fail(DLS_ERR_ARG, "adaptive.reserved must be 0");
  if (!std::isfinite(r.h_lo) || !std::isfinite(r.h_hi) || !(r.h_lo < r.h_hi))
    return fail(DLS_ERR_ARG, "the gate needs finite h_lo < h_hi (got %g, %g)", (double)r.h_lo, (double)r.h_hi);
  return DLS_OK;
}

dls::UncRule unc_rule(const dls_adaptive& r, int32_t V) {
  dls::UncRule u;
  u.measure = r.measure;
  u.inv_log_v = V > 1 ? (float)(1.0 / std::log((double)V)) : 0.f;
  u.maxprob_scale = V > 1 ? (float)((double)V / (double)(V - 1)) : 0.f;
  u.h_lo = r.h_lo;
  u.inv_width = (float)(1.0 / ((double)r.h_hi - (double)r.h_lo));
  return u;
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

dls_status check_head(const dls_local_head* h) {
  if (!h) return fail(DLS_ERR_ARG, "head is NULL");
  if (h->kind != DLS_HEAD_RNN && h->kind != DLS_HEAD_MARKOV) return fail(DLS_ERR_ARG, "unknown head kind %d", h->kind);
  const bool markov = h->kind == DLS_HEAD_MARKOV;
  if (!valid_dtype(enum_bits(h->dtype))) return fail(DLS_ERR_DTYPE, "unknown head dtype %d", enum_bits(h->dtype));
  if (h->V < 1 || h->V > (1 << 24)) return fail(DLS_ERR_SHAPE, "V=%d outside [1, 2^24]", h->V);
  if (!markov && (h->d < 8 || h->d > 16384 || h->d % 8))
    return fail(DLS_ERR_SHAPE, "d=%d must be a multiple of 8 in [8, 16384]", h->d);
  if (!markov && (h->H < 8 || h->H > 4096 || h->H % 8))
    return fail(DLS_ERR_SHAPE, "H=%d must be a multiple of 8 in [8, 4096]", h->H);
  if (h->r < 8 || h->r > 512 || h->r % 8)
    return fail(DLS_ERR_SHAPE, "r=%d must be a multiple of 8 in [8, 512]", h->r);
  const void* ps[5] = {h->emb, h->w_vocab, h->w_ih, h->w_hh, h->w_rank};
  const char* nm[5] = {"emb", "w_vocab", "w_ih", "w_hh", "w_rank"};
  for (int i = 0; i < (markov ? 2 : 5); ++i) {
    if (!ps[i]) return fail(DLS_ERR_ARG, "head.%s is NULL", nm[i]);
    if (!aligned(ps[i], 16)) return fail(DLS_ERR_ARG, "head.%s is not 16-byte aligned", nm[i]);
  }
  return DLS_OK;
}

// A head that dls_prepare_head accepts: a valid bf16 head with r in {32, 64, 128, 256} and, for
// the RNN head, H a multiple of 32.
dls_status check_preparable(const dls_local_head* head) {
  dls_status s = check_head(head);
  if (s != DLS_OK) return s;
  if (head->dtype != DLS_BF16) return fail(DLS_ERR_DTYPE, "only bf16 heads can be prepared");
  if (head->kind == DLS_HEAD_RNN && head->H % 32)
    return fail(DLS_ERR_SHAPE, "H=%d must be a multiple of 32 to prepare", head->H);
  if (!(head->r == 32 || head->r == 64 || head->r == 128 || head->r == 256))
    return fail(DLS_ERR_SHAPE, "r=%d must be 32, 64, 128 or 256 to prepare", head->r);
  return DLS_OK;
}

// The head as the kernels see it: a Markov head has no GRU (d = H = 0, no GRU tensors).
dls_local_head canon(const dls_local_head& h) {
  dls_local_head c = h;
  if (h.kind == DLS_HEAD_MARKOV) {
    c.d = 0;
    c.H = 0;
    c.w_ih = c.w_hh = c.w_rank = nullptr;
  }
  c.reserved = 0;
  return c;
}

}  // namespace

extern "C" {

const char* dls_status_string(dls_status s) {
  switch (enum_bits(s)) {
    case DLS_OK: return "DLS_OK";
    case DLS_ERR_ARG: return "DLS_ERR_ARG";
    case DLS_ERR_SHAPE: return "DLS_ERR_SHAPE";
    case DLS_ERR_DTYPE: return "DLS_ERR_DTYPE";
    case DLS_ERR_WORKSPACE: return "DLS_ERR_WORKSPACE";
    case DLS_ERR_DEVICE: return "DLS_ERR_DEVICE";
    case DLS_ERR_HIP: return "DLS_ERR_HIP";
  }
  return "DLS_UNKNOWN_STATUS";
}

const char* dls_last_error(void) { return g_last_error; }

int dls_abi_version(void) { return DLS_ABI_VERSION; }

size_t dls_combine_logits_workspace_size(int64_t rows, int32_t V) {
  if (rows <= 0 || V <= 0) return 0;
  const int parts = dls::combine_parts(rows, V);
  size_t b = (size_t)rows * sizeof(float);                       // per-row normaliser
  b = (b + 255) & ~(size_t)255;
  if (parts > 1) b += (size_t)rows * parts * sizeof(dls::Partial);
  return b;
}

dls_status dls_combine_logits(const void* long_logits, const void* short_logits, dls_dtype dtype_in,
                              const float* prior, int64_t rows, int32_t V, dls_fusion fusion,
                              int32_t* out_token, dls_row_stats* out_stats, float* out_scores,
                              void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  if (!valid_dtype(enum_bits(dtype_in))) return fail(DLS_ERR_DTYPE, "unknown dtype %d", enum_bits(dtype_in));
  const dls_dtype dtype = static_cast<dls_dtype>(enum_bits(dtype_in));
  if (rows < 0 || rows > (1 << 20)) return fail(DLS_ERR_SHAPE, "rows=%lld outside [0, 2^20]", (long long)rows);
  if (V < 1 || V > (1 << 24)) return fail(DLS_ERR_SHAPE, "V=%d outside [1, 2^24]", V);
  dls_status s = check_fusion(fusion);
  if (s != DLS_OK) return s;
  if (rows == 0) return DLS_OK;
  if (!long_logits || !short_logits || !out_token) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(long_logits, 16) || !aligned(short_logits, 16))
    return fail(DLS_ERR_ARG, "logits must be 16-byte aligned");
  if (!aligned(out_token, 4) || (prior && !aligned(prior, 4)) || (out_stats && !aligned(out_stats, 4)) ||
      (out_scores && !aligned(out_scores, 16)))
    return fail(DLS_ERR_ARG, "misaligned output or prior pointer");
  const size_t need = dls_combine_logits_workspace_size(rows, V);
  if (ws_bytes < need) return fail(DLS_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (need && (!workspace || !aligned(workspace, 16)))
    return fail(DLS_ERR_ARG, "workspace is NULL or not 16-byte aligned");
  if ((s = check_device()) != DLS_OK) return s;

  dls::CombineArgs a;
  a.long_logits = long_logits;
  a.short_logits = short_logits;
  a.dtype = dtype;
  a.prior = prior;
  a.rows = rows;
  a.V = V;
  a.wl = fusion.w_long;
  a.al = fusion.alpha;
  a.be = prior ? fusion.beta : 0.f;
  a.parts = dls::combine_parts(rows, V);
  a.norm = (float*)workspace;
  a.partials = (dls::Partial*)((char*)workspace + (((size_t)rows * sizeof(float) + 255) & ~(size_t)255));
  a.out_token = out_token;
  a.out_stats = out_stats;
  a.out_scores = out_scores;
  hipError_t e = dls::launch_combine(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "combine_logits launch");
  return DLS_OK;
}

size_t dls_prepare_head_size(const dls_local_head* head) {
  if (check_preparable(head) != DLS_OK) return 0;
  clear_error();
  return dls::prepared_layout(canon(*head)).total;
}

dls_status dls_prepare_head(const dls_local_head* head, void* prepared, size_t bytes, void* stream) {
  clear_error();
  dls_status s = check_preparable(head);
  if (s != DLS_OK) return s;
  if (!prepared || !aligned(prepared, 256)) return fail(DLS_ERR_ARG, "prepared buffer is NULL or not 256-byte aligned");
  const dls_local_head ch = canon(*head);
  const size_t need = dls::prepared_layout(ch).total;
  if (bytes < need) return fail(DLS_ERR_WORKSPACE, "prepared buffer %zu bytes < %zu required", bytes, need);
  if ((s = check_device()) != DLS_OK) return s;
  hipError_t e = dls::launch_prepare(ch, prepared, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "prepare_head launch");
  return DLS_OK;
}

size_t dls_draft_block_workspace_size(const dls_local_head* head, int32_t batch, int32_t B) {
  if (!head || batch <= 0 || B <= 0 || check_head(head) != DLS_OK) return 0;
  clear_error();
  const dls_local_head ch = canon(*head);
  // persistent region first (its header must start zero-filled), per-launch region after it,
  // then the partials of the adaptive-fusion pre-pass
  return dls::persist_workspace(ch, std::min<int32_t>(batch, dls::kMaxBatch), B).total +
         dls::draft_layout(ch, batch, B).total +
         align256(dls::uncertainty_workspace_bytes((int64_t)batch * B, ch.V));
}

size_t dls_long_uncertainty_workspace_size(int64_t rows, int32_t V) {
  if (rows <= 0 || V <= 0) return 0;
  return dls::uncertainty_workspace_bytes(rows, V);
}

dls_status dls_long_uncertainty(const void* long_logits, dls_dtype dtype_in, int64_t rows, int32_t V,
                                dls_adaptive rule, dls_row_uncertainty* out, void* workspace, size_t ws_bytes,
                                void* stream) {
  clear_error();
  if (!valid_dtype(enum_bits(dtype_in))) return fail(DLS_ERR_DTYPE, "unknown dtype %d", enum_bits(dtype_in));
  const dls_dtype dtype = static_cast<dls_dtype>(enum_bits(dtype_in));
  if (rows < 0 || rows > (1 << 24)) return fail(DLS_ERR_SHAPE, "rows=%lld outside [0, 2^24]", (long long)rows);
  if (V < 1 || V > (1 << 24)) return fail(DLS_ERR_SHAPE, "V=%d outside [1, 2^24]", V);
  dls_status s = check_rule(rule);
  if (s != DLS_OK) return s;
  if (rows == 0) return DLS_OK;
  if (!long_logits || !out) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(long_logits, 16)) return fail(DLS_ERR_ARG, "long_logits must be 16-byte aligned");
  if (!aligned(out, 4)) return fail(DLS_ERR_ARG, "out is misaligned");
  const size_t need = dls_long_uncertainty_workspace_size(rows, V);
  if (ws_bytes < need) return fail(DLS_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
  if (need && (!workspace || !aligned(workspace, 16)))
    return fail(DLS_ERR_ARG, "workspace is NULL or not 16-byte aligned");
  if ((s = check_device()) != DLS_OK) return s;
  dls::UncArgs a;
  a.long_logits = long_logits;
  a.dtype = dtype;
  a.rows = rows;
  a.V = V;
  a.rule = unc_rule(rule, V);
  a.partials = (float4*)workspace;
  a.out = out;
  hipError_t e = dls::launch_uncertainty(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "long_uncertainty launch");
  return DLS_OK;
}

}  // extern "C"

namespace {

// Checks of a prepared buffer that need no device access: its stated size.
dls_status check_prepared_size(const dls_local_head* head) {
  if (!head->prepared) return DLS_OK;
  const size_t need = dls::prepared_layout(canon(*head)).total;
  if (head->prepared_bytes < need)
    return fail(DLS_ERR_WORKSPACE, "head.prepared_bytes = %zu, but this head's prepared form needs %zu bytes",
                head->prepared_bytes, need);
  if (!aligned(head->prepared, 256)) return fail(DLS_ERR_ARG, "head.prepared is not 256-byte aligned");
  return DLS_OK;
}

// The drafting entry points.  noalloc: run in the current device's scratch array instead of
// the caller's workspace (workspace and ws_bytes are then ignored).
dls_status draft_impl(const dls_local_head* head, const void* long_logits, int long_dtype_bits,
                      const int32_t* last_token, const float* prior, int32_t batch, int32_t B, dls_fusion fusion,
                      const float* alphas, const float* betas, dls_sampling sampling, int32_t* out_tokens,
                      dls_row_stats* out_stats, void* workspace, size_t ws_bytes, void* stream,
                      bool noalloc = false, const dls_adaptive* rule = nullptr,
                      dls_row_uncertainty* out_unc = nullptr) {
  dls_status s = check_head(head);
  if (s != DLS_OK) return s;
  if ((s = check_prepared_size(head)) != DLS_OK) return s;
  if (!valid_dtype(long_dtype_bits)) return fail(DLS_ERR_DTYPE, "unknown long-logit dtype %d", long_dtype_bits);
  const dls_dtype long_dtype = static_cast<dls_dtype>(long_dtype_bits);
  if (batch < 0 || batch > 256) return fail(DLS_ERR_SHAPE, "batch=%d outside [0, 256]", batch);
  if (B < 0 || B > 64) return fail(DLS_ERR_SHAPE, "B=%d outside [0, 64]", B);
  if ((s = check_fusion(fusion)) != DLS_OK) return s;
  if (batch == 0 || B == 0) return DLS_OK;
  for (int j = 0; j < B; ++j) {
    if ((alphas && !std::isfinite(alphas[j])) || (betas && !std::isfinite(betas[j])))
      return fail(DLS_ERR_ARG, "per-position fusion weight %d is not finite", j);
  }
  const float T = sampling.temperature;
  if (sampling.reserved != 0) return fail(DLS_ERR_ARG, "sampling.reserved must be 0");
  if (!(T == 0.f || (T > 0.f && T <= 1e30f && std::isfinite(1.f / T))))
    return fail(DLS_ERR_ARG, "temperature %g must be 0 or a finite positive value with a finite inverse", (double)T);
  dls::Sampler smp;
  smp.inv_temp = T > 0.f ? 1.f / T : 0.f;
  smp.temp = T > 0.f ? T : 1.f;
  smp.seed_lo = (uint32_t)sampling.seed;
  smp.seed_hi = (uint32_t)(sampling.seed >> 32);
  smp.b0 = 0;
  const bool literal = (fusion.flags & DLS_FIRST_ROW_LONG_ONLY) != 0;
  if (!long_logits || !out_tokens || (!last_token && !literal))
    return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(long_logits, 16)) return fail(DLS_ERR_ARG, "long_logits must be 16-byte aligned");
  if ((last_token && !aligned(last_token, 4)) || !aligned(out_tokens, 4) || (prior && !aligned(prior, 4)) ||
      (out_stats && !aligned(out_stats, 4)))
    return fail(DLS_ERR_ARG, "misaligned vector argument");
  if (rule) {
    if ((s = check_rule(*rule)) != DLS_OK) return s;
    if (!out_unc || !aligned(out_unc, 4)) return fail(DLS_ERR_ARG, "out_uncertainty is NULL or misaligned");
  }
  const size_t need = dls_draft_block_workspace_size(head, batch, B);
  if (noalloc) {
    if (need > dls::kNoallocScratchBytes)
      return fail(DLS_ERR_WORKSPACE,
                  "dls_draft_block_noalloc: batch %d, B %d of this head need %zu bytes of scratch, more than the "
                  "library's %zu-byte array", batch, B, need, dls::kNoallocScratchBytes);
  } else {
    if (ws_bytes < need) return fail(DLS_ERR_WORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, need);
    if (!workspace || !aligned(workspace, 256))
      return fail(DLS_ERR_ARG, "workspace is NULL or not 256-byte aligned");
  }
  int cus = 0;
  if ((s = check_device(&cus)) != DLS_OK) return s;
  if (noalloc) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) workspace = dls::noalloc_scratch(dev, &e);
    if (e != hipSuccess) return hip_fail(e, "draft_block_noalloc scratch address");
    ws_bytes = dls::kNoallocScratchBytes;
    // a failed previous call on this scratch: restore it before this call uses it
    if ((e = dls::launch_scratch_guard(workspace, (hipStream_t)stream)) != hipSuccess)
      return hip_fail(e, "draft_block_noalloc scratch check");
  }

  const dls_local_head ch = canon(*head);
  // the persistent kernel runs at most kMaxBatch sequences per launch (below)
  const dls::PersistWorkspace pw = dls::persist_workspace(ch, std::min<int32_t>(batch, dls::kMaxBatch), B);
  // adaptive fusion: the gates of all batch * B rows first, stream-ordered before the draft
  if (rule) {
    dls::UncArgs ua;
    ua.long_logits = long_logits;
    ua.dtype = long_dtype;
    ua.rows = (int64_t)batch * B;
    ua.V = ch.V;
    ua.rule = unc_rule(*rule, ch.V);
    ua.partials = (float4*)((char*)workspace + pw.total + dls::draft_layout(ch, batch, B).total);
    ua.out = out_unc;
    hipError_t e = dls::launch_uncertainty(ua, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "draft_block_adaptive uncertainty launch");
  }
  if (head->prepared) {
    // A call of more than kMaxBatch sequences runs as consecutive launches of at most kMaxBatch
    // sequences each, on the same workspace and stream; every launch's plan is checked first.
    const int nfull = std::min<int32_t>(batch, dls::kMaxBatch);
    const int nlast = batch - (batch - 1) / dls::kMaxBatch * dls::kMaxBatch;   // the last launch's sequences
    const dls::PersistPlan pl = dls::persist_plan(ch, nfull, B, long_dtype, prior != nullptr, persist_groups(cus));
    const dls::PersistPlan pl_last = nlast == nfull ? pl
                                                    : dls::persist_plan(ch, nlast, B, long_dtype, prior != nullptr,
                                                                        persist_groups(cus));
    if (pl.ok && pl_last.ok) {
      const dls::PreparedLayout PL = dls::prepared_layout(ch);
      const char* pp = (const char*)head->prepared;
      char* ws = (char*)workspace;
      dls::PersistArgs pa;
      pa.prep = (const dls::PreparedHeader*)pp;
      pa.expect.magic = dls::kPreparedMagic;
      pa.expect.V = ch.V;
      pa.expect.d = ch.d;
      pa.expect.H = ch.H;
      pa.expect.r = ch.r;
      pa.expect.emb = ch.emb;
      pa.expect.w_ih = ch.w_ih;
      pa.expect.w_hh = ch.w_hh;
      pa.expect.w_vocab = ch.w_vocab;
      pa.T = (const float*)(pp + PL.off_T);
      pa.wv = (const uint4*)(pp + PL.off_wv);
      pa.whh = (const uint4*)(pp + PL.off_whh);
      pa.w_rank = (const dls::bf16_t*)ch.w_rank;
      pa.e_m = ch.kind == DLS_HEAD_MARKOV ? (const dls::bf16_t*)ch.emb : nullptr;
      pa.V = head->V;
      pa.H = ch.H;
      pa.r = head->r;
      pa.prior = prior;
      pa.B = B;
      pa.wl = fusion.w_long;
      for (int j = 0; j < 64; ++j) {
        pa.al_j[j] = j < B && alphas ? alphas[j] : fusion.alpha;
        pa.be_j[j] = !prior ? 0.f : (j < B && betas ? betas[j] : fusion.beta);
      }
      pa.literal = (fusion.flags & DLS_FIRST_ROW_LONG_ONLY) ? 1 : 0;
      pa.ordinary_launch = (fusion.flags & DLS_EXCLUSIVE_DEVICE) ? 1 : 0;
      pa.hdr = (uint32_t*)ws;
      // one copy of the wide h hand-off words: replicas (each GRU workgroup reading its own) cost
      // more in publish stores on the critical path than they saved in reads
      pa.hrep = 1;
      const size_t lsz = long_dtype == DLS_BF16 ? 2 : 4;
      for (int b0 = 0; b0 < batch; b0 += dls::kMaxBatch) {
        const int nb = std::min<int32_t>(dls::kMaxBatch, batch - b0);
        const dls::PersistPlan& plc = nb == nfull ? pl : pl_last;
        const dls::PersistWorkspace pwc = dls::persist_workspace(ch, nb, B);
        pa.NT = plc.NT;
        pa.NG = plc.NG;
        pa.rpg = plc.rpg;
        pa.cap_a = plc.cap_a;
        pa.gcap = plc.gcap;
        pa.rows_max = plc.rows_max;
        pa.lds_region_a = plc.lds_region_a;
        pa.batch = nb;
        pa.L = (const char*)long_logits + (size_t)b0 * B * ch.V * lsz;
        pa.last = last_token ? last_token + b0 : nullptr;
        pa.smp = smp;
        pa.smp.b0 = (uint32_t)b0;   // the noise of a sequence is keyed by its index in the call
        pa.unc = out_unc ? out_unc + (size_t)b0 * B : nullptr;
        pa.out_tokens = out_tokens + (size_t)b0 * B;
        pa.out_stats = out_stats ? out_stats + (size_t)b0 * B : nullptr;
        pa.keys = (uint64_t*)(ws + pwc.off_keys);
        pa.hbuf = (uint64_t*)(ws + pwc.off_h);
        pa.h32 = (uint32_t*)(ws + pwc.off_h32);
        pa.rbuf = (uint64_t*)(ws + pwc.off_rho);
        pa.stats = (uint64_t*)(ws + pwc.off_stats);
        pa.tokw = (uint64_t*)(ws + pwc.off_tokw);
        hipError_t e = dls::launch_persistent(pa, plc, long_dtype, (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "draft_block persistent launch");
      }
      return DLS_OK;
    }
  }

  dls::DraftArgs a;
  a.head = ch;
  a.long_logits = long_logits;
  a.long_dtype = long_dtype;
  a.last_token = last_token;
  a.prior = prior;
  a.batch = batch;
  a.B = B;
  a.f = fusion;
  if (!prior) a.f.beta = 0.f;
  a.out_tokens = out_tokens;
  a.out_stats = out_stats;
  a.ws = (char*)workspace + pw.total;
  a.lay = dls::draft_layout(ch, batch, B);
  a.alphas = alphas;
  a.betas = betas;
  a.smp = smp;
  a.unc = out_unc;
  hipError_t e = dls::launch_draft(a, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "draft_block launch");
  return DLS_OK;
}

}  // namespace

extern "C" {

dls_status dls_draft_block(const dls_local_head* head, const void* long_logits, dls_dtype long_dtype,
                           const int32_t* last_token, const float* prior, int32_t batch, int32_t B,
                           dls_fusion fusion, int32_t* out_tokens, dls_row_stats* out_stats, void* workspace,
                           size_t ws_bytes, void* stream) {
  clear_error();
  return draft_impl(head, long_logits, enum_bits(long_dtype), last_token, prior, batch, B, fusion, nullptr, nullptr,
                    dls_sampling{0.f, 0u, 0ull}, out_tokens, out_stats, workspace, ws_bytes, stream);
}

dls_status dls_draft_block_scheduled(const dls_local_head* head, const void* long_logits, dls_dtype long_dtype,
                                     const int32_t* last_token, const float* prior, int32_t batch, int32_t B,
                                     dls_fusion fusion, dls_fusion_schedule schedule, int32_t* out_tokens,
                                     dls_row_stats* out_stats, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  return draft_impl(head, long_logits, enum_bits(long_dtype), last_token, prior, batch, B, fusion, schedule.alpha,
                    schedule.beta, dls_sampling{0.f, 0u, 0ull}, out_tokens, out_stats, workspace, ws_bytes, stream);
}

dls_status dls_draft_block_sampled(const dls_local_head* head, const void* long_logits, dls_dtype long_dtype,
                                   const int32_t* last_token, const float* prior, int32_t batch, int32_t B,
                                   dls_fusion fusion, dls_fusion_schedule schedule, dls_sampling sampling,
                                   int32_t* out_tokens, dls_row_stats* out_stats, void* workspace, size_t ws_bytes,
                                   void* stream) {
  clear_error();
  return draft_impl(head, long_logits, enum_bits(long_dtype), last_token, prior, batch, B, fusion, schedule.alpha,
                    schedule.beta, sampling, out_tokens, out_stats, workspace, ws_bytes, stream);
}

dls_status dls_draft_block_adaptive(const dls_local_head* head, const void* long_logits, dls_dtype long_dtype,
                                    const int32_t* last_token, const float* prior, int32_t batch, int32_t B,
                                    dls_fusion fusion, dls_fusion_schedule schedule, dls_sampling sampling,
                                    dls_adaptive rule, dls_row_uncertainty* out_uncertainty, int32_t* out_tokens,
                                    dls_row_stats* out_stats, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  return draft_impl(head, long_logits, enum_bits(long_dtype), last_token, prior, batch, B, fusion, schedule.alpha,
                    schedule.beta, sampling, out_tokens, out_stats, workspace, ws_bytes, stream, false, &rule,
                    out_uncertainty);
}

dls_status dls_draft_block_noalloc(const dls_local_head* head, const void* long_logits, dls_dtype long_dtype,
                                   const int32_t* last_token, const float* prior, int32_t batch, int32_t B,
                                   dls_fusion fusion, int32_t* out_tokens, dls_row_stats* out_stats, void* stream) {
  clear_error();
  return draft_impl(head, long_logits, enum_bits(long_dtype), last_token, prior, batch, B, fusion, nullptr, nullptr,
                    dls_sampling{0.f, 0u, 0ull}, out_tokens, out_stats, nullptr, 0, stream, true);
}

dls_status dls_draft_block_error(const void* workspace, size_t ws_bytes, int32_t* out_error, void* stream) {
  clear_error();
  if (!out_error || !aligned(out_error, 4)) return fail(DLS_ERR_ARG, "out_error is NULL or misaligned");
  if (workspace && (ws_bytes < 256 || !aligned(workspace, 256)))
    return fail(DLS_ERR_WORKSPACE, "a drafting workspace has at least 256 bytes and is 256-byte aligned");
  dls_status s = check_device();
  if (s != DLS_OK) return s;
  hipError_t e = hipSuccess;
  if (!workspace) {
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) workspace = dls::noalloc_scratch(dev, &e);
    if (e != hipSuccess) return hip_fail(e, "draft_block_error scratch address");
  }
  e = dls::launch_copy_word((const uint32_t*)workspace + 1, out_error, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "draft_block_error launch");
  return DLS_OK;
}

int dls_draft_block_path(const dls_local_head* head, int32_t batch, int32_t B, dls_dtype long_dtype,
                         int has_prior) {
  clear_error();
  if (check_head(head) != DLS_OK || check_prepared_size(head) != DLS_OK || !valid_dtype(enum_bits(long_dtype)) ||
      batch < 1 || batch > 256 || B < 1 || B > 64)
    return -1;
  if (!head->prepared) return 0;
  int cus = 0;
  if (check_device(&cus) != DLS_OK) return -1;
  const int nfull = std::min<int32_t>(batch, dls::kMaxBatch);
  const int nlast = batch - (batch - 1) / dls::kMaxBatch * dls::kMaxBatch;
  const dls::PersistPlan pl = dls::persist_plan(canon(*head), nfull, B, long_dtype, has_prior != 0, persist_groups(cus));
  const dls::PersistPlan pl_last = dls::persist_plan(canon(*head), nlast, B, long_dtype, has_prior != 0,
                                                     persist_groups(cus));
  if (!pl.ok || !pl_last.ok) fail(DLS_OK, "%s", pl.ok ? pl_last.why : pl.why);
  return pl.ok && pl_last.ok ? 1 : 0;
}

dls_status dls_unigram_log_prior(const int32_t* tokens, int64_t n, int32_t V, float smoothing, uint64_t* out_counts,
                                 float* out_log_prior, void* stream) {
  clear_error();
  if (n < 0 || n > ((int64_t)1 << 40)) return fail(DLS_ERR_SHAPE, "n=%lld outside [0, 2^40]", (long long)n);
  if (V < 1 || V > (1 << 24)) return fail(DLS_ERR_SHAPE, "V=%d outside [1, 2^24]", V);
  if (!(smoothing >= 0.f) || !std::isfinite(smoothing)) return fail(DLS_ERR_ARG, "smoothing must be finite and >= 0");
  if (!out_counts || !out_log_prior || (n > 0 && !tokens)) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(out_counts, 8) || !aligned(out_log_prior, 4) || (tokens && !aligned(tokens, 4)))
    return fail(DLS_ERR_ARG, "misaligned pointer");
  dls_status s = check_device();
  if (s != DLS_OK) return s;
  hipError_t e = dls::launch_unigram_prior(tokens, n, V, smoothing, out_counts, out_log_prior, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "unigram_log_prior launch");
  return DLS_OK;
}

dls_status dls_accept_len(const int32_t* draft, const int32_t* target, int32_t batch, int32_t B, int32_t* out_len,
                          void* stream) {
  clear_error();
  if (batch < 0 || batch > (1 << 24)) return fail(DLS_ERR_SHAPE, "batch=%d outside [0, 2^24]", batch);
  if (B < 0 || B > 4096) return fail(DLS_ERR_SHAPE, "B=%d outside [0, 4096]", B);
  if (batch == 0) return DLS_OK;
  if (!out_len || (B > 0 && (!draft || !target))) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(out_len, 4) || (draft && !aligned(draft, 4)) || (target && !aligned(target, 4)))
    return fail(DLS_ERR_ARG, "misaligned pointer");
  dls_status s = check_device();
  if (s != DLS_OK) return s;
  hipError_t e = dls::launch_accept(draft, target, batch, B, out_len, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "accept_len launch");
  return DLS_OK;
}

dls_status dls_measure_read(const void* buf, size_t bytes, uint32_t* out, void* stream) {
  clear_error();
  if (bytes == 0 || bytes % 16 != 0) return fail(DLS_ERR_SHAPE, "bytes=%zu must be a positive multiple of 16", bytes);
  if (!buf || !out) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(buf, 16) || !aligned(out, 4)) return fail(DLS_ERR_ARG, "misaligned pointer");
  dls_status s = check_device();
  if (s != DLS_OK) return s;
  static_assert(dls::kMeasureReadGroups == DLS_MEASURE_READ_WORDS, "checksum word count");
  hipError_t e = dls::launch_measure_read(buf, bytes, out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "measure_read launch");
  return DLS_OK;
}

dls_status dls_measure_mfma(int32_t groups, int32_t iters, float x, float* out, void* stream) {
  clear_error();
  if (groups < 1 || groups > 65536) return fail(DLS_ERR_SHAPE, "groups=%d outside [1, 65536]", groups);
  if (iters < 1 || iters > (1 << 18)) return fail(DLS_ERR_SHAPE, "iters=%d outside [1, 2^18]", iters);
  if ((int64_t)groups * iters > ((int64_t)1 << 24))
    return fail(DLS_ERR_SHAPE, "groups x iters = %lld above 2^24", (long long)groups * iters);
  int ex = 0;
  if (!std::isfinite(x) || std::frexp(x, &ex) != 0.5f || ex < -19 || ex > 1)
    return fail(DLS_ERR_ARG, "x must be a power of two in [2^-20, 1]");
  if (!out) return fail(DLS_ERR_ARG, "required pointer is NULL");
  if (!aligned(out, 4)) return fail(DLS_ERR_ARG, "misaligned pointer");
  dls_status s = check_device();
  if (s != DLS_OK) return s;
  hipError_t e = dls::launch_measure_mfma(groups, iters, x, out, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "measure_mfma launch");
  return DLS_OK;
}

}  // extern "C"
