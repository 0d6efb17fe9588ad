// Holds on preloader images for a staged restore that copies each chunk image
// to the device as soon as it is staged, while the request's other files are
// still being read (Sec. 6.5: a demand load claims what is staged and joins
// reads in progress). Internal to libkvx.so.
#pragma once

#include <stdint.h>

#include <atomic>
#include <string>
#include <vector>

#include "kvx.h"

namespace kvx {

// Whether the pool is pinned (host-to-device copies may read it directly).
bool preload_pinned(const kvx_preloader* p);

// Hold the distinct files `paths` (all or none), in order, as a fetch does,
// without waiting: the files not yet staged are read as demand work in this
// order. One opaque handle per path, valid until preload_unhold.
// KVX_ENOMEM / KVX_EIO as for kvx_preload_fetch.
kvx_status preload_hold(kvx_preloader* p, const std::vector<std::string>& paths,
                        std::vector<void*>* handles);

// The image of a held file: *image and *size once staged; *image null if not
// yet staged and !wait. With wait, blocks until it is staged (KVX_ECLOSED if
// *cancel becomes true meanwhile). KVX_EIO if the file failed.
kvx_status preload_image(kvx_preloader* p, void* handle, bool wait,
                         const std::atomic<bool>* cancel, uint8_t** image, int64_t* size);

// Mark a held file's staged image as not to be used again (it does not match
// what the holder expected): it is dropped once nobody holds it, and the next
// hold reads the file again.
void preload_discard(kvx_preloader* p, void* handle);

// Drop the holds taken by preload_hold.
void preload_unhold(kvx_preloader* p, const std::vector<void*>& handles);

}  // namespace kvx
