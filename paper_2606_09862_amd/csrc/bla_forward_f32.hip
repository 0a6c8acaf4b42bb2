// float32 operands: v_mfma_f32_16x16x4_f32 (the float32 I/O path keeps float32 everywhere).
#include "bla_forward_inst.h"
BLA_DEFINE_DISPATCH(float, f32)
