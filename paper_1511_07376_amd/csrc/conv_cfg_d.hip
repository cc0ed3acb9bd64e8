// Instantiations of the convolution kernel for configurations 11, 12, 13.
#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {

CNN_CONV_DEFINE(11, 2, 4, 2, 2, 16, 1, 2)
CNN_CONV_DEFINE(12, 1, 2, 3, 2, 16, 1, 2)
CNN_CONV_DEFINE(13, 2, 1, 2, 2, 16, 1, 2)

}  // namespace conv
}  // namespace cnn
