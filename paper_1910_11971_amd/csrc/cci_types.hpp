// Plain host/device types shared by the launchers and the kernels.
#pragma once

#include <stdint.h>

namespace cci {

// Geometry of the GEMM operand A: row n of A is sample n (FC) or output
// pixel n of an NHWC convolution read through implicit im2col, with column
// c = (kh*KW + kw)*Cin + cin.
struct ConvGeom {
  int32_t H, W, Cin, KH, KW, sh, sw, ph, pw, Ho, Wo;
};

}  // namespace cci
