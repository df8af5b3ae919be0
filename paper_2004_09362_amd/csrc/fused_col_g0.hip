// fused_col_g0.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 2, 10, ..., 122 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<2>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<2>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<2>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<10>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<10>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<10>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<18>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<18>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<18>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<26>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<26>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<26>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<34>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<34>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<34>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<42>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<42>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<42>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<50>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<50>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<50>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<58>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<58>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<58>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<66>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<66>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<66>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<74>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<74>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<74>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<82>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<82>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<82>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<90>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<90>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<90>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<98>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<98>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<98>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<106>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<106>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<106>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<114>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<114>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<114>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<122>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<122>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<122>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
