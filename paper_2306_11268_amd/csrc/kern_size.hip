// One FFT size of the pass kernels; compiled once per supported size with
// -DLR_FFT_N=<size> so the sizes build in parallel.
#include "kernels_impl.hpp"

#ifndef LR_FFT_N
#error "define LR_FFT_N"
#endif

namespace lr {
template hipError_t launch_fr_n<LR_FFT_N>(PassKind, Axis, const PassArgs&, hipStream_t);
template int slots_fr_n<LR_FFT_N>(PassKind, Axis, bool);
template int tile_fr_n<LR_FFT_N>(PassKind, Axis, bool);
template hipError_t launch_as_n<LR_FFT_N>(AsPassKind, const PassArgs&, hipStream_t);
template hipError_t prep_as_n<LR_FFT_N>(const float2*, float2*, float, int, hipStream_t);
template TileShape shape_n<LR_FFT_N>();
template SlotMap slot_map_n<LR_FFT_N>();
template hipError_t launch_field_fwd_n<LR_FFT_N>(const FieldArgs&, hipStream_t);
}  // namespace lr
