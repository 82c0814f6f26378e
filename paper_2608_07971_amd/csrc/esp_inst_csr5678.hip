// Instances of the fused CSR kernels for R = 5, 6, 7, 8 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_CSR_DECL(5, )
ESP_CSR_DECL(6, )
ESP_CSR_DECL(7, )
ESP_CSR_DECL(8, )

}  // namespace esp
