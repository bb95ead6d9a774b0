"""MI355X-native Oaken KV-cache quantization and decode attention (HIP, gfx950).

The compute path lives in the C-ABI library ``liboaken.so`` built from ``csrc/``;
``paper_2503_18599_amd.binding`` marshals torch tensors into it.  Importing this
package does not load the library.
"""
