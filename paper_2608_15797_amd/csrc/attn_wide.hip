// The helper context kernels of three and four row blocks (48 to 64 query
// rows of the candidates sharing a context), compiled apart from attn.hip so
// that the build can give this translation unit alone the matrix-core
// accumulators in vector registers (-mllvm -amdgpu-mfma-vgpr-form=1). Their
// accumulators (up to 128 floats per lane) then stay put between key chunks:
// with them in accumulator registers the compiler copied them to and from
// vector registers on every chunk, around the rarely taken rescale.
#define KVR_ATTN_WIDE 1
#include "attn.hip"
