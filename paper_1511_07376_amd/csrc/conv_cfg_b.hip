// Instantiations of the convolution kernel for configurations 4, 5, 6, 7.
#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {

CNN_CONV_DEFINE(4, 1, 4, 2, 1, 16, 1, 2)
CNN_CONV_DEFINE(5, 1, 4, 2, 1, 32, 1, 2)
CNN_CONV_DEFINE(6, 1, 4, 3, 1, 16, 1, 2)
CNN_CONV_DEFINE(7, 1, 4, 3, 1, 32, 1, 2)

}  // namespace conv
}  // namespace cnn
