// bfloat16 operands: v_mfma_f32_16x16x32_bf16 with float32 accumulation.
#include "bla_forward_inst.h"
BLA_DEFINE_DISPATCH(bf16, bf16)
