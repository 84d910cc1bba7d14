"""MOSAIC hot path on MI355X: masked Z_{2^32} products, mask/unmask passes and
the random Hadamard rotation, as HIP kernels behind the C ABI of
include/mosaic.h. Importing the package loads nothing; the binding
(``paper_2607_29221_amd.mosaic``) loads libmosaic.so on first use."""
