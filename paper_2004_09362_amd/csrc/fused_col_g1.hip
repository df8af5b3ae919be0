// fused_col_g1.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 3, 11, ..., 123 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<3>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<3>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<3>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<11>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<11>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<11>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<19>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<19>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<19>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<27>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<27>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<27>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<35>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<35>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<35>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<43>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<43>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<43>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<51>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<51>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<51>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<59>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<59>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<59>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<67>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<67>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<67>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<75>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<75>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<75>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<83>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<83>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<83>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<91>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<91>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<91>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<99>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<99>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<99>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<107>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<107>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<107>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<115>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<115>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<115>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<123>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<123>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<123>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
