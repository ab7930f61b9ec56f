"""MI355X (gfx950) speculative diffusion sampling with block verification.

The native library is loaded lazily on first use (see _lib.py); importing the
package does not touch the GPU.
"""
