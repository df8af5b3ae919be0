// fused_col_g3.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 5, 13, ..., 125 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<5>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<5>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<5>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<13>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<13>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<13>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<21>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<21>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<21>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<29>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<29>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<29>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<37>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<37>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<37>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<45>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<45>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<45>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<53>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<53>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<53>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<61>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<61>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<61>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<69>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<69>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<69>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<77>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<77>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<77>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<85>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<85>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<85>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<93>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<93>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<93>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<101>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<101>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<101>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<109>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<109>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<109>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<117>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<117>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<117>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<125>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<125>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<125>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
