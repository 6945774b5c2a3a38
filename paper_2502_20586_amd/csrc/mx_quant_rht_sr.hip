// Instantiations of the quantiser for the paper's method (RHT + SR, 16-bit
// dither), every g.

#include "mx_quant_impl.h"

namespace mx {
namespace quant {

int launch_rht_sr(const QuantJobs& jobs, int g, bool kt, hipStream_t stream) {
  return kt ? launch_jobs_mode<true, 16, true>(jobs, g, stream) : launch_jobs_mode<true, 16, false>(jobs, g, stream);
}

}  // namespace quant
}  // namespace mx
