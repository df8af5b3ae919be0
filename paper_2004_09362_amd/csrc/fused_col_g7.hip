// fused_col_g7.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 9, 17, ..., 121 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<9>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<9>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<9>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<17>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<17>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<17>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<25>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<25>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<25>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<33>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<33>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<33>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<41>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<41>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<41>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<49>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<49>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<49>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<57>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<57>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<57>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<65>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<65>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<65>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<73>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<73>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<73>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<81>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<81>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<81>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<89>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<89>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<89>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<97>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<97>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<97>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<105>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<105>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<105>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<113>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<113>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<113>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<121>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<121>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<121>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
