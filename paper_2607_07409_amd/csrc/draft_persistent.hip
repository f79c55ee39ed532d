// Host side of the persistent drafting kernel: the launch plan (tile ownership, LDS
// budget), the workspace layout and the dispatch to the instantiations (one translation
// unit per rank size and decoding mode, built in parallel).
#include "draft_persistent.hpp"

namespace dls {

extern template hipError_t launch_persistent_kk<4, false>(const PersistArgs&, int, size_t, dls_dtype, hipStream_t);
extern template hipError_t launch_persistent_kk<8, false>(const PersistArgs&, int, size_t, dls_dtype, hipStream_t);
extern template hipError_t launch_persistent_kk<4, true>(const PersistArgs&, int, size_t, dls_dtype, hipStream_t);
extern template hipError_t launch_persistent_kk<8, true>(const PersistArgs&, int, size_t, dls_dtype, hipStream_t);

PersistPlan persist_plan(const dls_local_head& h, int32_t batch, int32_t B, dls_dtype long_dtype, bool prior,
                         int G) {
  PersistPlan pl;
  pl.ok = false;
  const int KK = h.r / 32;
  // r = 128 or 256: the vocabulary tiles of a wave fill its 256 AGPRs without spills
  if (h.dtype != DLS_BF16 || h.r % 32 || !(KK == 4 || KK == 8) || h.H % 32 ||
      batch < 1 || batch > kMaxBatch || B < 1 || B > 64 || h.V >= (1 << 24) || G < 1 || G > kMaxG) {
    pl.why = "shape outside the persistent kernel's range";
    return pl;
  }
  const bool markov = h.kind == DLS_HEAD_MARKOV;   // no GRU workgroups
  const int NG = markov ? 0 : h.H / 16;
  if (!markov && h.H > kStageK && h.H % kStageK) {
    pl.why = "H above 256 must be a multiple of 256";
    return pl;
  }
  if (!markov && (NG > G || h.r % NG || h.r / NG > 16)) {
    pl.why = "hidden size / rank do not split over the workgroups";
    return pl;
  }
  pl.G = G;
  pl.NG = NG;
  pl.rpg = markov ? 0 : h.r / NG;
  pl.NT = (h.V + 15) / 16;
  pl.cap_a = 4 * (kOps / KK);
  const size_t esz = long_dtype == DLS_BF16 ? 2 : 4;
  const int ll_slots = batch < 16 ? batch : 16;
  // LDS need of the tile split with gcap tiles per GRU workgroup (0: a GRU workgroup's tiles
  // exceed its AGPRs)
  auto lds_need = [&](int gcap, int* rows_out, size_t* region_out) -> size_t {
    int rows_max = 0, nl_max = 0;
    for (int w = 0; w < G; ++w) {
      int t0, n;
      persist_tile_range(w, G, NG, pl.NT, pl.cap_a, gcap, &t0, &n);
      rows_max = std::max(rows_max, 16 * n);
      if (w >= NG) nl_max = std::max(nl_max, n - std::min(n, pl.cap_a));
      else if (n > pl.cap_a) return 0;
    }
    const size_t region_gru = markov ? 0 : (size_t)3 * (h.H / 32) * 1024 + (size_t)pl.rpg * h.H * 2;
    const size_t region_tiles = (size_t)nl_max * KK * 1024;
    const size_t region_a = (std::max(region_gru, region_tiles) + 15) & ~(size_t)15;
    size_t lds = region_a + (((size_t)ll_slots * rows_max * esz + 15) & ~(size_t)15);
    if (prior) lds += (size_t)rows_max * 4;
    lds += (size_t)2 * kPlane * 2 + (size_t)16 * pl.rpg * 16 + (size_t)((batch + 15) / 16) * 16 * 48 * 4 +
           (size_t)4 * 16 * sizeof(Partial) + (size_t)kMaxBatch * 8 + (size_t)kMaxBatch * 4 + 16 * 4 + 16;
    *rows_out = rows_max;
    *region_out = region_a;
    return lds;
  };
  // Narrow batches: the GRU workgroups reach their vocabulary tiles about 2 us after the others
  // (they compute W_hh h and stage rho first), so they take three quarters of a full AGPR load
  // and the others hold the surplus in LDS, which narrow batches leave free; the share grows
  // back toward a full load while the others' LDS would overflow.  Wide batches: a full load.
  int gcap = (batch <= kNarrowBatch && !markov) ? (3 * pl.cap_a + 3) / 4 : pl.cap_a;
  int rows_max = 0;
  size_t region_a = 0, lds = lds_need(gcap, &rows_max, &region_a);
  while ((lds == 0 || lds > kMaxLds) && gcap < pl.cap_a) lds = lds_need(++gcap, &rows_max, &region_a);
  if (lds == 0) {
    pl.why = "vocabulary tiles exceed the GRU workgroups' AGPRs";
    return pl;
  }
  pl.gcap = gcap;
  pl.lds_region_a = region_a;
  pl.rows_max = rows_max;
  pl.lds = lds;
  if (lds > kMaxLds) {
    pl.why = "per-workgroup LDS need exceeds 160 KiB";
    return pl;
  }
  pl.ok = true;
  return pl;
}

PersistWorkspace persist_workspace(const dls_local_head& h, int32_t batch, int32_t B) {
  PersistWorkspace L;
  size_t o = 256;                                     // header: epoch, error word
  L.off_keys = o;
  o += (size_t)2 * 2 * kMaxBatch * kMaxG * 8;
  // the two sets of 32-bit h words sit at a fixed offset with a fixed size, whatever the
  // batch, B or H of a call: their 8-bit tags must never meet words another layout left there
  L.off_h32 = o;
  o += 2 * kH32Set * 4;
  L.off_h = o;
  o += (size_t)2 * batch * h.H * 8;
  L.off_rho = o;
  o += (size_t)kRhoCopies * 2 * batch * h.r * 8;
  L.off_tokw = o;
  o += (size_t)2 * kMaxBatch * 8;
  L.off_stats = o;
  o += (size_t)B * batch * kMaxG * kStatWords * 8;
  L.total = (o + 255) & ~(size_t)255;
  return L;
}

namespace {
__global__ void k_copy_word(const uint32_t* src, int32_t* dst) {
  *dst = (int32_t)__hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
}  // namespace

hipError_t launch_copy_word(const uint32_t* src, int32_t* dst, hipStream_t st) {
  k_copy_word<<<1, 1, 0, st>>>(src, dst);
  return hipGetLastError();
}

hipError_t launch_persistent(const PersistArgs& pa, const PersistPlan& pl, dls_dtype long_dtype, hipStream_t st) {
  const bool sample = pa.smp.inv_temp != 0.f;
  switch (pa.r / 32) {
    case 4:
      return sample ? launch_persistent_kk<4, true>(pa, pl.G, pl.lds, long_dtype, st)
                    : launch_persistent_kk<4, false>(pa, pl.G, pl.lds, long_dtype, st);
    case 8:
      return sample ? launch_persistent_kk<8, true>(pa, pl.G, pl.lds, long_dtype, st)
                    : launch_persistent_kk<8, false>(pa, pl.G, pl.lds, long_dtype, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace dls
