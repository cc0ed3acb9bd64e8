// Instantiations of the convolution kernel for configurations 0, 1, 2, 3.
#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {

CNN_CONV_DEFINE(0, 2, 2, 2, 2, 16, 1, 2)
CNN_CONV_DEFINE(1, 2, 2, 2, 2, 32, 1, 2)
CNN_CONV_DEFINE(2, 4, 1, 1, 2, 16, 1, 2)
CNN_CONV_DEFINE(3, 4, 1, 1, 2, 32, 1, 2)

}  // namespace conv
}  // namespace cnn
