// Run-time dispatch of the Elastic Shadow Pricing launchers on R (and on
// the lanes per job of the dense kernel).  The fused kernels are instantiated
// in the esp_inst_*.hip files; the small kernels here.
#include "esp_kernels.hpp"

namespace esp {

#define ESP_EXTERN_DENSE(RR) ESP_DENSE_DECL(RR, extern)
#define ESP_EXTERN_CSR(RR) ESP_CSR_DECL(RR, extern)
ESP_FUSED_LAUNCHERS(ESP_EXTERN_DENSE)
ESP_FUSED_LAUNCHERS(ESP_EXTERN_CSR)

hipError_t launch_dense(int R, int lpj, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_dense_r<RR>(lpj, a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_dense_persistent(int R, int lpj, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_dense_coop_r<RR>(lpj, a, B, false, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_dense_resident(int R, int lpj, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_dense_coop_r<RR>(lpj, a, B, true, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_gather(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_gather_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_update(int R, const KArgs &a, const double *demand_in, int B, hipStream_t s) {
#define CALL(RR) launch_update_r<RR>(a, demand_in, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_prepare(int R, const KArgs &a, const double *lam, double *canon, int B, hipStream_t s) {
#define CALL(RR) launch_prepare_r<RR>(a, lam, canon, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_finish(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_finish_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_csr_persistent(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_csr_coop_r<RR>(a, B, false, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_csr_resident(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_csr_coop_r<RR>(a, B, true, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_csr(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_csr_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}


}  // namespace esp
