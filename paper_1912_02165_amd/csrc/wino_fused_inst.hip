// One instantiation of the fused kernel (wino_ws.h) per object file: the build
// compiles this file once for every entry of WINO_FUSED_BLOCKINGS, with
// WS_M, WS_TB, WS_FS and WS_CSP defined, so the kernels compile in parallel.
#include "wino_ws.h"

#if !defined(WS_M) || !defined(WS_TB) || !defined(WS_FS) || !defined(WS_CSP)
#error "compile with -DWS_M=<m> -DWS_TB=<tb> -DWS_FS=<fs> -DWS_CSP=<csp>"
#endif

namespace wino {

template hipError_t launch_ws_t<WS_M, WS_TB, WS_FS, WS_CSP>(const Geometry &, const float *, const float *,
                                                            float *, bool, int, int, const SplitBuffers &,
                                                            hipStream_t);

}  // namespace wino
