// layer_fp32.hip - the per-layer launch sequence instantiated for float I/O with float
// MFMA operands (its own translation unit, compiled in parallel with the others).
#include "layer.hpp"

namespace still {
template still_status run_layer<float, float>(const still_config*, const Dims&, const Plan&, char*,
                                          const still_layer_weights*, const void*, const void*, const double*,
                                          bool, void*, void*, hipStream_t);
}  // namespace still
