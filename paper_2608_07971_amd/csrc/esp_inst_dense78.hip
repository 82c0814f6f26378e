// Instances of the fused dense kernels for R = 7, 8 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_DENSE_DECL(7, )
ESP_DENSE_DECL(8, )

}  // namespace esp
