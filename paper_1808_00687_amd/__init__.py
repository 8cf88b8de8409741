"""MI355X-native WFST Viterbi beam decoder (frame- and label-synchronous)
with state-level lattice generation, after Z. Chen, "Linguistic Search
Optimization for Deep Learning Based LVCSR" (Interspeech 2018).

The decoder is the C-ABI library ``libwfstdec.so`` (HIP kernels for gfx950);
``paper_1808_00687_amd.wfstdec`` is its thin Python binding.  Importing this
package does not load the library; ``workloads`` holds the seeded synthetic
inputs.
"""
