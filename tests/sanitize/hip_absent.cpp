// Stand-ins for the HIP runtime calls and the kernel launches the host
// runtime makes, for a build of its host-only paths without a GPU: a
// host-only context and a no-device scheduler must never reach the device,
// so every one of these stops the program at once.
#include <hip/hip_runtime_api.h>

#include "rb.h"

#include <cstdio>
#include <cstdlib>

[[noreturn]] static void reached(const char* f) {
  std::fprintf(stderr, "device call %s reached from a host-only path\n", f);
  std::abort();
}

extern "C" {
hipError_t hipEventCreate(hipEvent_t*) { reached("hipEventCreate"); }
hipError_t hipEventCreateWithFlags(hipEvent_t*, unsigned) { reached("hipEventCreateWithFlags"); }
hipError_t hipEventDestroy(hipEvent_t) { reached("hipEventDestroy"); }
hipError_t hipEventElapsedTime(float*, hipEvent_t, hipEvent_t) { reached("hipEventElapsedTime"); }
hipError_t hipEventQuery(hipEvent_t) { reached("hipEventQuery"); }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { reached("hipEventRecord"); }
hipError_t hipEventSynchronize(hipEvent_t) { reached("hipEventSynchronize"); }
hipError_t hipFree(void*) { reached("hipFree"); }
hipError_t hipGetDeviceCount(int*) { reached("hipGetDeviceCount"); }
hipError_t hipHostFree(void*) { reached("hipHostFree"); }
hipError_t hipHostMalloc(void**, size_t, unsigned) { reached("hipHostMalloc"); }
hipError_t hipMalloc(void**, size_t) { reached("hipMalloc"); }
hipError_t hipMemcpy(void*, const void*, size_t, hipMemcpyKind) { reached("hipMemcpy"); }
hipError_t hipMemcpyAsync(void*, const void*, size_t, hipMemcpyKind, hipStream_t) { reached("hipMemcpyAsync"); }
hipError_t hipMemset(void*, int, size_t) { reached("hipMemset"); }
hipError_t hipSetDevice(int) { reached("hipSetDevice"); }
hipError_t hipStreamCreateWithFlags(hipStream_t*, unsigned) { reached("hipStreamCreateWithFlags"); }
hipError_t hipStreamDestroy(hipStream_t) { reached("hipStreamDestroy"); }
hipError_t hipStreamSynchronize(hipStream_t) { reached("hipStreamSynchronize"); }
hipError_t hipStreamWaitEvent(hipStream_t, hipEvent_t, unsigned) { reached("hipStreamWaitEvent"); }

rb_status rb_k_route(void*, int32_t, const rb_k_batch*, int32_t, const rb_k_req*, int32_t, const int32_t*, int64_t,
                     int32_t, int32_t, int32_t, rb_k_row*, int32_t, int64_t, int32_t*) {
  reached("rb_k_route");
}
rb_status rb_k_assemble(void*, const rb_k_row*, int32_t, int32_t, int32_t, const float*, int64_t, int32_t, void*,
                        int32_t, int32_t, float, int32_t*) {
  reached("rb_k_assemble");
}
rb_status rb_k_embbag(void*, const rb_k_row*, int32_t, const int32_t*, const int32_t*, int64_t, const void* const*,
                      int32_t, int64_t, int32_t, const float*, int32_t, void*, int32_t, float, int32_t*) {
  reached("rb_k_embbag");
}
rb_status rb_k_embbag_dedup(void*, const rb_k_row*, int32_t, const int32_t*, const int32_t*, int64_t,
                            const void* const*, int32_t, int64_t, int32_t, const float*, int32_t, void*, int32_t, float,
                            int32_t*) {
  reached("rb_k_embbag_dedup");
}
rb_status rb_k_gemm_bf16(void*, const void*, int32_t, const void*, int32_t, const float*, void*, int32_t, int32_t,
                         int32_t, int32_t, int32_t, int32_t) {
  reached("rb_k_gemm_bf16");
}
rb_status rb_k_gemm_f32(void*, const float*, int32_t, const float*, int32_t, const float*, float*, int32_t, int32_t,
                        int32_t, int32_t, int32_t, const rb_k_row*, int32_t) {
  reached("rb_k_gemm_f32");
}
rb_status rb_k_head(void*, const rb_k_row*, int32_t, const void*, int32_t, const void*, float, int32_t, int32_t,
                    float*) {
  reached("rb_k_head");
}
rb_status rb_k_gemm_bf16_rows(void*, const void*, int32_t, const void*, int32_t, const float*, int32_t, int32_t,
                              int32_t, int32_t, const rb_k_row*, int32_t, float*) {
  reached("rb_k_gemm_bf16_rows");
}
rb_status rb_k_gemm_f32_rows(void*, const float*, int32_t, const float*, int32_t, const float*, int32_t, int32_t,
                             int32_t, int32_t, const rb_k_row*, int32_t, float*) {
  reached("rb_k_gemm_f32_rows");
}
rb_status rb_k_gemm_head(void*, const void*, int32_t, const void*, int32_t, const float*, int32_t, int32_t, int32_t,
                         const rb_k_row*, const void*, float, int32_t, float*) {
  reached("rb_k_gemm_head");
}
rb_status rb_k_mlp_tail(void*, const rb_k_row*, int32_t, const void*, int32_t, int32_t, const void*, int32_t,
                        const float*, const void*, int32_t, const float*, const void*, float, int32_t, float*) {
  reached("rb_k_mlp_tail");
}
rb_status rb_k_seqpool(void*, const rb_k_row*, int32_t, int32_t, int64_t, const float*, int32_t, int32_t,
                       const float*, const float*, int32_t, int32_t, float*) {
  reached("rb_k_seqpool");
}
rb_status rb_k_split(void*, const rb_k_row*, int32_t, const float*, int32_t, int32_t, float*) {
  reached("rb_k_split");
}
}

void rb_scrub_caches(hipStream_t, const void*, size_t, unsigned*) { reached("rb_scrub_caches"); }
void rb_fill_padding_rows(hipStream_t, rb_k_row*, int64_t) { reached("rb_fill_padding_rows"); }
rb_status rb_static_scratch_setup(int) { reached("rb_static_scratch_setup"); }
void* rb_static_scratch(int) { reached("rb_static_scratch"); }
