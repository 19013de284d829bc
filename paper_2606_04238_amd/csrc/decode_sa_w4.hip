// Instantiations of the stand-alone decode kernels (decode_standalone.h)
// for one code width, in a translation unit of their own.
#include "decode_standalone.h"

namespace qmlp {

template hipError_t launch_gateup_bits<4, false, 256>(BatchArgs, int, int, hipStream_t);
template hipError_t launch_down_bits<4, 256>(BatchArgs, int, int, hipStream_t);
template hipError_t launch_down_bits<4, 1024>(BatchArgs, int, int, hipStream_t);

template hipError_t launch_gateup_routed_bits<4, false>(BatchArgs, int, int, unsigned long long*, unsigned*,
                                                     hipStream_t);

}  // namespace qmlp
