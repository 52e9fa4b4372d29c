// Buffers the host stand-ins of the kernel launchers accept as device memory.
#pragma once
#include <stddef.h>

void stub_register(const void* p, size_t bytes);
void stub_unregister(const void* p);
long stub_launches();   // launcher and runtime calls made so far
// Called by abi.cpp (built with HSPEC_HOST_SANITIZE) for every region it cuts from a workspace.
void hspec_host_carve(const void* p, size_t bytes);
