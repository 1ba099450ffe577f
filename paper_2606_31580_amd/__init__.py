"""MI355X-native (gfx950) decode + confidence-probe hot path of LASER.

The compute path is the C-ABI library ``liblaser.so`` (hand-written HIP kernels);
``paper_2606_31580_amd.laser`` is its thin ctypes binding.  Importing the
package does not load the library.
"""
