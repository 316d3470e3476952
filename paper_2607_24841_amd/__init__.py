"""libnmdlm: the N-MDLM block-denoising step on MI355X (gfx950).

The compute lives in the HIP library ``libnmdlm.so`` (C ABI in
``include/nmdlm.h``); ``binding`` marshals torch tensors to it.  Importing the
package does not load the library; the first call does, and raises if the
library is not built.
"""
