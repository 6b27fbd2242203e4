"""MI355X (gfx950) sparse spiking BPTT: HIP kernels behind the C ABI of include/snn.h.

`snn` is the ctypes binding of libsnn.so; `pipeline` chains its calls over a whole
fully connected LIF network; `build` compiles the library with hipcc.
"""
