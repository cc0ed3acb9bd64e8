"""MI355X-native forward pass of trained CNNs (conv, FC, ReLU, max/avg pooling, LRN).

The compute path is the C-ABI library ``libcnn.so`` built from ``csrc/`` (HIP for
gfx950); ``paper_1511_07376_amd.cnn`` is its thin Python binding.  Importing this
package loads nothing native; ``paper_1511_07376_amd.cnn`` loads the library on
import and raises if it is missing.
"""

__all__ = ["workloads", "cnn"]
