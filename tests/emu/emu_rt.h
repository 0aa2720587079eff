// Interface between the emulated kernels (compiled for the host) and the emulator runtime.
#pragma once
#include <cstdint>

struct EmuDim { unsigned x, y, z; };
struct EmuThread { EmuDim tid; int lane, wave, flat; };

extern "C" {
extern EmuThread* emu_cur;         // the running emulated thread
extern EmuDim emu_blockIdx, emu_blockDim, emu_gridDim;
// deposit `n` bytes for the wave collective at call site `site`; returns the wave's 64 slots
// of 64 bytes (slot l = lane l's deposit) once every live lane of the wave has arrived, and
// the mask of lanes that took part
const unsigned char* emu_wave_op(const void* in, int n, int site, uint64_t* mask);
void emu_syncthreads(int site);
void emu_run_grid(const char* name, EmuDim grid, EmuDim block, void (*entry)(void*), void* ctx);
void emu_note(const char* fmt, ...);
// the kernel module's LDS (all __shared__ arrays), poisoned before every block
void emu_set_lds(char* begin, char* end);
}
