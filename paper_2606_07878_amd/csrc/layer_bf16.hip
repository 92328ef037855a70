// layer_bf16.hip - the per-layer launch sequence instantiated for bf16 I/O with f16
// MFMA operands (its own translation unit, compiled in parallel with the others).
#include "layer.hpp"

namespace still {
template still_status run_layer<bf16, f16>(const still_config*, const Dims&, const Plan&, char*,
                                          const still_layer_weights*, const void*, const void*, const double*,
                                          bool, void*, void*, hipStream_t);
}  // namespace still
