/* Host BMI2 parallel-bit-deposit, used only to pin the oracle's pdep. */
#include <immintrin.h>
#include <stdint.h>

uint32_t host_pdep_u32(uint32_t a, uint32_t mask) { return _pdep_u32(a, mask); }
