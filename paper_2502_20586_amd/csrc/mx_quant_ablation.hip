// Instantiations of the quantiser for the ablation modes of Table 2: SR
// without the RHT, RHT + round to nearest, round to nearest.

#include "mx_quant_impl.h"

namespace mx {
namespace quant {

namespace {
template <bool KT>
int launch_kt(const QuantJobs& jobs, int g, QuantMode mode, hipStream_t stream) {
  switch (mode) {
    case QuantMode::kSr: return launch_jobs_mode<false, 16, KT>(jobs, g, stream);
    case QuantMode::kRhtNr: return launch_jobs_mode<true, 0, KT>(jobs, g, stream);
    case QuantMode::kNr: return launch_jobs_mode<false, 0, KT>(jobs, g, stream);
    default: return -1;
  }
}
}  // namespace

int launch_ablation(const QuantJobs& jobs, int g, bool kt, QuantMode mode, hipStream_t stream) {
  return kt ? launch_kt<true>(jobs, g, mode, stream) : launch_kt<false>(jobs, g, mode, stream);
}

}  // namespace quant
}  // namespace mx
