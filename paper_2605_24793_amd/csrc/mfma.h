// Matrix-core step shared by the two forms of the head's first layer (head.hip's
// LDS-tiled GEMM over the mismatch rows and slot_gemm.h's register-fed GEMM over every
// decision slot): one 64-byte k-step of a 16 x 16 fp32 tile.
//
// Operand layout: lane l supplies row (l % 16) of A and column (l % 16) of B for the
// 16-byte k-piece owned by lane group l / 16, and receives D[4*(l/16) + j][l % 16] in
// accumulator element j.  A and B take the same k-piece per lane, so the order of k
// inside an instruction is immaterial.
#pragma once

#include <hip/hip_runtime.h>

#include "launch.h"
#include "rowstat.h"

namespace cospec {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float floatx4;

// bf16: one v_mfma_f32_16x16x32_bf16 (8 elements per lane); fp32: four
// v_mfma_f32_16x16x4_f32 (one element per lane each).
template <int DT> __device__ inline floatx4 mma(u32x4 a, u32x4 b, floatx4 c);
template <> __device__ inline floatx4 mma<kBF16>(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <> __device__ inline floatx4 mma<kF32>(u32x4 a, u32x4 b, floatx4 c) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[j]), __uint_as_float(b[j]), c, 0, 0, 0);
    return c;
}

}  // namespace cospec
