"""MI355X-native environment-plus-policy step of GPU-native DeepMimic-style
imitation training (InstantMimic, arXiv 2609.09821).

The compute path lives in the HIP library built from csrc/ (C ABI declared in
include/instantmimic.h); `binding` is a thin ctypes layer over it and `synth`
makes the seeded synthetic inputs.  Submodules are imported lazily so that
`synth` can be used without loading the HIP library.
"""
