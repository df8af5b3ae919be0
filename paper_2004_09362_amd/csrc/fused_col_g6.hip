// fused_col_g6.hip -- instantiations of the column-fused kernels
// (bandwidth-optimal, shifted/latency-optimal and rank-slot) for P = 8, 16, ..., 128 (every 8th P; the eight files share the
// work evenly and compile in parallel).
#include "fused_col.hpp"

namespace ar {

template int launch_fused_bo<8>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<8>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<8>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<16>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<16>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<16>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<24>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<24>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<24>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<32>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<32>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<32>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<40>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<40>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<40>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<48>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<48>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<48>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<56>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<56>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<56>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<64>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<64>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<64>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<72>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<72>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<72>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<80>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<80>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<80>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<88>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<88>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<88>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<96>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<96>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<96>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<104>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<104>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<104>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<112>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<112>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<112>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<120>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<120>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<120>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_bo<128>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_mid<128>(const ColArgs&, int, int, bool, int, void*);
template int launch_fused_rot<128>(const ColArgs&, int, int, bool, int, void*);

}  // namespace ar
