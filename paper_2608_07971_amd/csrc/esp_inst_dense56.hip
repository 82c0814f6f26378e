// Instances of the fused dense kernels for R = 5, 6 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_DENSE_DECL(5, )
ESP_DENSE_DECL(6, )

}  // namespace esp
