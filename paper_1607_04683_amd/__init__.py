"""MI355X (gfx950) quantized LSTM acoustic-model inference.

Implements the 8-bit uniform linear quantization scheme of Alvarez,
Prabhavalkar and Bakhtin, "On the efficient representation and execution of
deep acoustic models" (Interspeech 2016), as hand-written HIP kernels behind a
C ABI (include/qlstm.h).  The Python module `qlstm` is a thin ctypes binding
over that library; PyTorch is used only for device memory and streams.
"""
