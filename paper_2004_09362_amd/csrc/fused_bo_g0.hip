// fused_bo_g0.hip -- instantiations of the column-fused bandwidth-optimal
// kernel for P = 2, 10, ..., 122 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_bo.hpp"

namespace ar {

template int launch_fused_bo<2>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<10>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<18>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<26>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<34>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<42>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<50>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<58>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<66>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<74>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<82>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<90>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<98>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<106>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<114>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<122>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
