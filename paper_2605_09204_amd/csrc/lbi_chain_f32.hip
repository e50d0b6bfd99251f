// Chain-kernel instantiations for one arithmetic mode (one translation unit
// per mode, so the library builds in parallel).
#include "lbi_chain.hpp"

namespace lbi {

hipError_t launch_chain_f32(const ChainLaunch &c) { return launch_chain<kF32>(c); }

}  // namespace lbi
