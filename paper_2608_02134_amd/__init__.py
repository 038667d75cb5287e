"""MI355X-native GMC boundary operator (Grounded Message Coreset pruning).

The operator itself lives in the HIP/C++ shared library ``libgmc.so`` built
from ``csrc/``; ``binding`` marshals arguments to its C-ABI.  Importing this
package does not load the library; ``binding.lib()`` does, and raises if the
library has not been built.
"""
__all__ = ["binding", "synth"]
