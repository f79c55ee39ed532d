// Instantiations of the persistent drafting kernel for rank r = 256 (sampled decoding).
#include "draft_persistent.hpp"

namespace dls {
template hipError_t launch_persistent_kk<8, true>(const PersistArgs&, int, size_t, dls_dtype,
                                                       hipStream_t);
}  // namespace dls
