// Chain-kernel instantiations for one arithmetic mode (one translation unit
// per mode, so the library builds in parallel).
#include "lbi_chain.hpp"

namespace lbi {

hipError_t launch_chain_bf16r1(const ChainLaunch &c) { return launch_chain<kBF16R1>(c); }

}  // namespace lbi
