// The per-GPU static scratch array of the allocation-free attention entry
// point (headkv_decode_attn_noalloc): room for the merge words of a chunked
// attention launch, so that the call needs no workspace.  It is zero when the
// library loads, and every launch leaves the words it uses zero again.
#pragma once

#include <cstddef>

namespace headkv {

constexpr size_t kScratchBytes = (size_t)4 << 20;

// Device address of the array on the current GPU (looked up once per GPU,
// with that GPU current); returns a hipError_t as an int.
int scratch_address(void** ptr);

}  // namespace headkv
