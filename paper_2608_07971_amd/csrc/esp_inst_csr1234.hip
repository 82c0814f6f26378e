// Instances of the fused CSR kernels for R = 1, 2, 3, 4 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_CSR_DECL(1, )
ESP_CSR_DECL(2, )
ESP_CSR_DECL(3, )
ESP_CSR_DECL(4, )

}  // namespace esp
