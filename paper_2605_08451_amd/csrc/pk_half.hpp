// pk_half.hpp -- complex arithmetic on packed fp16 pairs (low half real, high half
// imaginary) with the packed-half ALU instructions.
//
// In these VOP3P instructions op_sel picks the source halves that feed the low
// result, op_sel_hi those that feed the high result, and neg_lo / neg_hi negate a
// source in the low / high result, so swaps and conjugations cost nothing.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace rubiconv {

__device__ __forceinline__ uint32_t h2_bits(float re, float im) {  // round to nearest even
    return __builtin_bit_cast(uint32_t, __float22half2_rn(make_float2(re, im)));
}

// bf16 of f rounded to nearest even, in the low 16 bits (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// (bf16(lo), bf16(hi)) rounded to nearest even: one v_cvt_pk_bf16_f32.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf2_bits(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// a * b
__device__ __forceinline__ uint32_t cmul_h2(uint32_t a, uint32_t b) {
    uint32_t t;
    asm("v_pk_mul_f16 %0, %1, %2 op_sel_hi:[0,1]" : "=v"(t) : "v"(a), "v"(b));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1] neg_lo:[1,0,0]"
        : "+v"(t) : "v"(a), "v"(b));
    return t;
}

// a * conj(b)
__device__ __forceinline__ uint32_t cmul_conj_h2(uint32_t a, uint32_t b) {
    uint32_t t;
    asm("v_pk_mul_f16 %0, %1, %2 op_sel_hi:[0,1] neg_hi:[0,1]" : "=v"(t) : "v"(a), "v"(b));
    asm("v_pk_fma_f16 %0, %1, %2, %0 op_sel:[1,1,0] op_sel_hi:[1,0,1]" : "+v"(t) : "v"(a), "v"(b));
    return t;
}

}  // namespace rubiconv
