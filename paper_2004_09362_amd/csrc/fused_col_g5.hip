// fused_col_g5.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 7, 15, ..., 127 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<7>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<7>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<7>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<15>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<15>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<15>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<23>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<23>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<23>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<31>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<31>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<31>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<39>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<39>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<39>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<47>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<47>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<47>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<55>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<55>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<55>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<63>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<63>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<63>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<71>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<71>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<71>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<79>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<79>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<79>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<87>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<87>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<87>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<95>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<95>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<95>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<103>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<103>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<103>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<111>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<111>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<111>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<119>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<119>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<119>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<127>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<127>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<127>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
