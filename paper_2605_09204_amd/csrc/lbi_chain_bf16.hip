// Chain-kernel instantiations for one arithmetic mode (one translation unit
// per mode, so the library builds in parallel).
#include "lbi_chain.hpp"

namespace lbi {

hipError_t launch_chain_bf16(const ChainLaunch &c) { return launch_chain<kBF16>(c); }

}  // namespace lbi
