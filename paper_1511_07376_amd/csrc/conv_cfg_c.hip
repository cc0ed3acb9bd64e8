// Instantiations of the convolution kernel for configurations 8, 9, 10.
#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {

CNN_CONV_DEFINE(8, 1, 4, 1, 1, 16, 1, 2)
CNN_CONV_DEFINE(9, 2, 2, 1, 1, 16, 1, 2)
CNN_CONV_DEFINE(10, 2, 2, 1, 1, 32, 1, 2)

}  // namespace conv
}  // namespace cnn
