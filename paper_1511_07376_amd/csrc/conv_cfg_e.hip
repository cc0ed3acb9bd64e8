// Instantiations of the convolution kernel for configurations 14 and 15.
#include "conv_igemm_kernel.h"

namespace cnn {
namespace conv {

CNN_CONV_DEFINE(14, 2, 2, 1, 1, 16, 2, 2)
CNN_CONV_DEFINE(15, 2, 1, 2, 2, 16, 2, 2)

}  // namespace conv
}  // namespace cnn
