// Instances of the fused dense kernels for R = 1, 2 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_DENSE_DECL(1, )
ESP_DENSE_DECL(2, )

}  // namespace esp
