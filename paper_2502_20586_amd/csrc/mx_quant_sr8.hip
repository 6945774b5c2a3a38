// Instantiations of the quantiser for the cheaper-noise variant (RHT + SR,
// 8-bit dither), g >= 64.

#include "mx_quant_impl.h"

namespace mx {
namespace quant {

int launch_rht_sr8(const QuantJobs& jobs, int g, bool kt, hipStream_t stream) {
  return kt ? launch_jobs_mode<true, 8, true>(jobs, g, stream) : launch_jobs_mode<true, 8, false>(jobs, g, stream);
}

}  // namespace quant
}  // namespace mx
