// Host-only stand-ins for the kernel launchers of libmosaic, linked with the
// ABI layer (abi.cpp) in the sanitizer build of tests/test_abi_sanitize.py.
// The driver only makes calls that validation must reject, so any launcher
// reached is a failure: each one counts the call and reports an error.
#include "../paper_2607_29221_amd/csrc/internal.h"

int g_launches = 0;

namespace mosaic {
#define STUB { ++g_launches; return hipErrorInvalidValue; }
hipError_t launch_mask(const MaskLaunch&, hipStream_t) STUB
hipError_t launch_signs(const RngArgs&, int64_t, int8_t*, hipStream_t) STUB
hipError_t launch_sparse_csr_count(const RngArgs&, int64_t, int64_t, int64_t*, hipStream_t) STUB
hipError_t launch_sparse_csr_fill(const RngArgs&, int64_t, int64_t, const int64_t*, int32_t*, uint32_t*,
                                  hipStream_t) STUB
hipError_t launch_sparse_gather_rows(int64_t, const int64_t*, const int32_t*, const uint32_t*, const uint32_t*,
                                     int64_t, int64_t, uint32_t*, int64_t, int, hipStream_t) STUB
hipError_t launch_sparse_stream_gather_rows(const RngArgs&, int64_t, int64_t, const uint32_t*, int64_t, int64_t,
                                            uint32_t*, int64_t, int, hipStream_t) STUB
hipError_t launch_sparse_gather_cols(int64_t, int64_t, const int64_t*, const int32_t*, const uint32_t*,
                                     const uint32_t*, int64_t, uint32_t*, int64_t, int, const Dequant&,
                                     hipStream_t) STUB
hipError_t launch_weighted_sample(const RngArgs&, int64_t, int64_t, uint32_t*, int64_t, int8_t*, int64_t,
                                  hipStream_t) STUB
hipError_t launch_weighted_csr_count(int64_t, int64_t, int64_t*, hipStream_t) STUB
hipError_t launch_weighted_csr_fill(const RngArgs&, int64_t, int64_t, const int64_t*, int32_t*, uint32_t*,
                                    hipStream_t) STUB
hipError_t launch_mfma_probe(int, int64_t, int32_t*, int64_t*, hipStream_t) STUB
hipError_t launch_count_mismatches(const uint32_t*, int64_t, const uint32_t*, int64_t, int64_t, int64_t, int64_t*,
                                   hipStream_t, bool) STUB
hipError_t launch_clear_check(uint32_t*, int64_t, int64_t, int64_t, int64_t*, hipStream_t) STUB
hipError_t launch_ring_gemm(const GemmLaunch&, EpilogueKind, hipStream_t) STUB
hipError_t launch_ring_gemm_skinny(const GemmLaunch&, EpilogueKind, hipStream_t) STUB
hipError_t launch_ring_gemm_words_b(const GemmLaunch&, EpilogueKind, hipStream_t) STUB
hipError_t launch_unmask_words_a(const GemmLaunch&, hipStream_t) STUB
hipError_t launch_unmask_elementwise(const GemmLaunch&, hipStream_t) STUB
hipError_t launch_hadamard(const float*, int64_t, float*, int64_t, int64_t, int64_t, int, const int8_t*, int,
                           hipStream_t) STUB
bool hadamard28_supported(int log2_block) { return log2_block >= 8 && log2_block <= 10; }
hipError_t launch_hadamard28(const float*, int64_t, float*, int64_t, int64_t, int, const int8_t*, int,
                             hipStream_t) STUB
bool rotate_quantize_mask_supported(int log2_block) { return log2_block >= 10 && log2_block <= 14; }
hipError_t launch_rotate_quantize_mask(const float*, int64_t, int64_t, int64_t, int, const int8_t*, int32_t,
                                       const uint32_t*, int64_t, const RngArgs*, int8_t*, int64_t, float*,
                                       hipStream_t) STUB
hipError_t launch_quantize_rows(const float*, int64_t, int64_t, int64_t, int32_t, int32_t*, int64_t, int8_t*,
                                int64_t, float*, hipStream_t) STUB
#undef STUB
}  // namespace mosaic
