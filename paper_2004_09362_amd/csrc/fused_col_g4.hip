// fused_col_g4.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 6, 14, ..., 126 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<6>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<6>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<6>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<14>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<14>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<14>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<22>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<22>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<22>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<30>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<30>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<30>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<38>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<38>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<38>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<46>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<46>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<46>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<54>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<54>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<54>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<62>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<62>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<62>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<70>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<70>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<70>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<78>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<78>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<78>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<86>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<86>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<86>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<94>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<94>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<94>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<102>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<102>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<102>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<110>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<110>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<110>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<118>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<118>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<118>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<126>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<126>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<126>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
