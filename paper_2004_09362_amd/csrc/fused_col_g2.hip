// fused_col_g2.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 4, 12, ..., 124 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<4>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<4>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<4>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<12>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<12>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<12>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<20>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<20>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<20>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<28>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<28>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<28>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<36>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<36>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<36>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<44>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<44>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<44>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<52>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<52>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<52>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<60>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<60>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<60>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<68>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<68>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<68>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<76>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<76>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<76>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<84>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<84>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<84>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<92>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<92>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<92>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<100>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<100>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<100>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<108>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<108>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<108>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<116>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<116>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<116>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<124>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<124>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<124>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
