// Host-only stand-ins for the kernel launchers of libqx, so that the C-ABI front end
// (qx_api.cpp: validation and the host packers) builds with g++ and the address,
// undefined-behaviour and thread sanitizers. Every device call reports QX_E_HIP.
#include "../../paper_2505_07531_amd/csrc/qx_internal.h"

namespace qx {
int launch_dequant(const qx_desc*, const void*, int, void*, hipStream_t) { return QX_E_HIP; }
int launch_gemv(const qx_desc*, const void*, const uint16_t*, uint16_t*, hipStream_t) { return QX_E_HIP; }
int launch_gemm(const qx_desc*, const void*, int, const uint16_t*, uint16_t*, hipStream_t) { return QX_E_HIP; }
int launch_gemv_a8(const qx_desc*, const void*, const uint16_t*, uint16_t*, hipStream_t) { return QX_E_HIP; }
int launch_quantize_a8(int, int, const uint16_t*, int8_t*, float*, hipStream_t) { return QX_E_HIP; }
int launch_gemm_a8(const qx_desc*, const void*, int, const int8_t*, const float*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
int launch_gemv_a8_multi(const qx_desc*, const void*, int, const int8_t*, const float*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
int launch_gemv_lut_a8(const qx_desc*, const void*, const uint16_t*, uint16_t*, hipStream_t) { return QX_E_HIP; }
int launch_gemm_lut_a8(const qx_desc*, const void*, int, const int8_t*, const float*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
int launch_gemv_a8q(const qx_desc*, const void*, const int8_t*, const float*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
bool gemv_multi_applies(const qx_desc*, int) { return false; }
int launch_gemv_multi(const qx_desc*, const void*, int, const uint16_t*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
bool gemm_skinny_applies(const qx_desc*, int) { return false; }
int launch_gemm_skinny(const qx_desc*, const void*, int, const uint16_t*, uint16_t*, hipStream_t) {
  return QX_E_HIP;
}
}  // namespace qx
