/* Link script of the weight-specialised kernel template: the default layout,
 * plus the section .jitbody placed after everything else, so that it forms
 * the last loadable segment, alone, at the highest address. The library
 * replaces that segment's contents with generated code at run time. */
SECTIONS {
  .jitbody : { *(.jitbody) }
} INSERT AFTER .bss;
