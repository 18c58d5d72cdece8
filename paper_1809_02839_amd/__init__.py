"""MI355X-native SpecTrain pipeline-stage step.

The compute path is libspectrain.so (hand-written HIP for gfx950), reached
through the C ABI declared in include/spectrain.h. This package holds the thin
ctypes binding (`native`), the one-forward-one-backward driver that simulates
a K-stage pipeline on one GPU (`pipeline`) and the in-tree build (`build`).
Importing the package loads nothing; the library is opened on first use and a
missing library raises instead of falling back to anything else.
"""
