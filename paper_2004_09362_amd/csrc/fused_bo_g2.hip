// fused_bo_g2.hip -- instantiations of the column-fused bandwidth-optimal
// kernel for P = 4, 12, ..., 124 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_bo.hpp"

namespace ar {

template int launch_fused_bo<4>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<12>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<20>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<28>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<36>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<44>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<52>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<60>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<68>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<76>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<84>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<92>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<100>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<108>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<116>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<124>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
