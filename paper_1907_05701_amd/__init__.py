"""MI355X learner step of H-ADPSGD: BLSTM forward/BPTT, softmax cross-entropy,
super-learner gradient reduction and the ADPSGD local update, as a C-ABI HIP
library (``libadpsgd_blstm.so``) with a thin ctypes binding.

Importing the package does not load the library; ``binding.lib()`` does, and
raises if the library is missing."""
