// Instances of the fused dense kernels for R = 3, 4 (compiled on their own, in
// parallel with the other instance files).
#include "esp_kernels.hpp"

namespace esp {

ESP_DENSE_DECL(3, )
ESP_DENSE_DECL(4, )

}  // namespace esp
