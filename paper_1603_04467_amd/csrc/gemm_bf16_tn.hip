// The TN layout of the 16-bit whole-tile MatMul (weight gradients:
// dW = H^T dY), compiled from gemm_bf16.hip in a translation unit of its own:
// the build gives this unit the max-ILP machine scheduler, measured faster
// for this layout (its 16 waves interleave two transposing reads per
// fragment with the MFMAs) and slower for NN and NT.
#define TFD_GEMM_BF16_TN_UNIT 1
#include "gemm_bf16.hip"
