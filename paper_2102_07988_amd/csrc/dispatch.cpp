// Kernel selection: the bf16 fast kernels where they cover the shape, the
// generic kernels otherwise (and for the fp32 validation mode).
#include "tp_common.hpp"
#include "tp_kernels.hpp"

namespace tp {

hipError_t attn_fwd_generic(int dtype, const AttnArgs& a, hipStream_t s);
hipError_t attn_bwd_generic(int dtype, const AttnArgs& a, hipStream_t s);

hipError_t gemm_mfma_bf16(const GemmArgs& a, hipStream_t s);
hipError_t gemm_dma_bf16(const GemmArgs& a, hipStream_t s);

hipError_t gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  clear_stale_error();
  if (dtype == DT_BF16) {
    hipError_t e = gemm_dma_bf16(a, s);
    if (e != hipErrorNotSupported) return e;
    e = gemm_mfma_bf16(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  // fp16 operands have no generic kernel (the stage only asks for them where
  // the matrix-core kernels apply)
  if (a.in_f16) return hipErrorNotSupported;
  return gemm_generic(dtype, a, s);
}

hipError_t attn_fwd_mfma_bf16(const AttnArgs& a, hipStream_t s);
hipError_t attn_bwd_mfma_bf16(const AttnArgs& a, hipStream_t s);

hipError_t attn_fwd(int dtype, const AttnArgs& a, hipStream_t s) {
  clear_stale_error();
  if (dtype == DT_BF16) {
    const hipError_t e = attn_fwd_mfma_bf16(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  if (a.f16) return hipErrorNotSupported;
  return attn_fwd_generic(dtype, a, s);
}

hipError_t attn_bwd(int dtype, const AttnArgs& a, hipStream_t s) {
  clear_stale_error();
  if (dtype == DT_BF16) {
    const hipError_t e = attn_bwd_mfma_bf16(a, s);
    if (e != hipErrorNotSupported) return e;
  }
  if (a.f16) return hipErrorNotSupported;
  return attn_bwd_generic(dtype, a, s);
}

}  // namespace tp
